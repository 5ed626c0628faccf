// Adaptive KV cache manager: where every node's K/V lives over a schedule of calls (micro-batches).
//
// Sec. 5.1 (adaptive block allocation): a node of the prefix tree -- one shared contiguous token
// segment -- gets one block of exactly its length, so shared prefixes are stored once and no
// slot is padding; the fixed-page alternative (block_size > 0) rounds each node up to pages.
// Sec. 5.2 (dynamic block caching): a block's reference count is the number of samples that will
// read it; each call's backward decrements it by the call's samples that read it, and at zero the
// block's gradient accumulators are complete and its slots are released.  Under memory pressure a
// cached block that the current call does not need is evicted, the one whose next use lies
// farthest ahead first; a later call that needs it again gets it back in a fresh block (its K/V
// recomputed by the caller, its dK/dV accumulators restarted at zero).
//
// The manager is host-only planning: it decides, for every call, which nodes are computed there
// (internal), which are read from the cache (external), and the pool slots of each, and it emits
// the events the caller acts on.  psattn_kvm_call_desc turns a call into the tree descriptor of
// psattn_tree_create.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <map>
#include <new>
#include <string>
#include <vector>

#include "psattn.h"

namespace psattn {
psattn_status set_error(psattn_status st, const char* msg);
}

namespace {

psattn_status kfail(psattn_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return psattn::set_error(st, buf);
}

// Free extents of the pool, best fit, coalesced on release.
class SlotAllocator {
 public:
  explicit SlotAllocator(int64_t n) {
    if (n > 0) free_[0] = n;
  }
  bool alloc(int64_t n, int64_t* base) {
    auto best = free_.end();
    for (auto it = free_.begin(); it != free_.end(); ++it)
      if (it->second >= n && (best == free_.end() || it->second < best->second)) best = it;
    if (best == free_.end()) return false;
    *base = best->first;
    const int64_t rest = best->second - n, at = best->first + n;
    free_.erase(best);
    if (rest > 0) free_[at] = rest;
    used_ += n;
    return true;
  }
  void release(int64_t base, int64_t n) {
    used_ -= n;
    auto it = free_.emplace(base, n).first;
    auto nx = std::next(it);
    if (nx != free_.end() && it->first + it->second == nx->first) {
      it->second += nx->second;
      free_.erase(nx);
    }
    if (it != free_.begin()) {
      auto pv = std::prev(it);
      if (pv->first + pv->second == it->first) {
        pv->second += it->second;
        free_.erase(it);
      }
    }
  }
  int64_t used() const { return used_; }

 private:
  std::map<int64_t, int64_t> free_;
  int64_t used_ = 0;
};

struct Page {
  int64_t base;
  int32_t cap, len;
};

psattn_kvm_event event(psattn_kvm_event_kind kind, int node, const std::vector<Page>& pages) {
  psattn_kvm_event ev;
  ev.kind = kind;
  ev.node = node;
  ev.num_blocks = (int32_t)pages.size();
  ev.capacity = pages.front().cap;
  ev.base = pages.front().base;
  return ev;
}

struct CallPlan {
  std::vector<int32_t> nodes;             // forest nodes on the call's sample paths, in order
  std::vector<char> ext;                  // cached from an earlier call
  std::vector<std::vector<Page>> pages;   // each node's blocks during the call
  std::vector<int32_t> sample_end;        // forest endpoint of each of the call's samples
  std::vector<psattn_kvm_event> before, after;
  int64_t used = 0;                       // slots in use during the call
  // descriptor arrays (psattn_kvm_call_desc)
  std::vector<int32_t> d_parent, d_seg, d_blk_ptr, d_end;
  std::vector<int64_t> d_row_off;
  std::vector<psattn_block> d_blocks;
};

}  // namespace

struct psattn_kvm {
  int32_t N = 0, S = 0, C = 0;
  int64_t capacity = 0;
  std::vector<CallPlan> calls;
  psattn_kvm_stats stats{};
};

namespace {

psattn_status build(psattn_kvm* m, const int32_t* parent, const int32_t* seg_len, const int32_t* sample_end,
                    const int32_t* call_of_sample, const psattn_kvm_opts& o) {
  const int N = m->N, S = m->S;
  std::vector<int64_t> off(N, 0);
  for (int i = 0; i < N; ++i) {
    if (parent[i] < -1 || parent[i] >= i)
      return kfail(PSATTN_E_INVALID_TREE, "parent[%d] = %d: a parent must precede its child (or be -1)", i, parent[i]);
    if (seg_len[i] < 1) return kfail(PSATTN_E_INVALID_TREE, "seg_len[%d] = %d: segments must be non-empty", i, seg_len[i]);
    off[i] = parent[i] < 0 ? 0 : off[parent[i]] + seg_len[parent[i]];
  }
  int C = 0;
  for (int s = 0; s < S; ++s) {
    if (sample_end[s] < 0 || sample_end[s] >= N)
      return kfail(PSATTN_E_INVALID_TREE, "sample_end[%d] = %d out of range", s, sample_end[s]);
    if (call_of_sample[s] < 0) return kfail(PSATTN_E_INVALID_ARG, "call_of_sample[%d] = %d is negative", s, call_of_sample[s]);
    C = std::max(C, call_of_sample[s] + 1);
  }
  m->C = C;
  m->calls.assign(C, {});
  // reference counts (samples reading each node) and, per call, how many of its samples read it
  std::vector<int32_t> refcount(N, 0);
  std::vector<std::vector<int32_t>> reads(C, std::vector<int32_t>(N, 0));
  for (int s = 0; s < S; ++s) {
    CallPlan& cp = m->calls[call_of_sample[s]];
    cp.sample_end.push_back(sample_end[s]);
    for (int n = sample_end[s]; n >= 0; n = parent[n]) {
      refcount[n]++;
      reads[call_of_sample[s]][n]++;
    }
  }
  for (int i = 0; i < N; ++i)
    if (refcount[i] == 0) return kfail(PSATTN_E_INVALID_TREE, "node %d lies on no sample path", i);
  for (int c = 0; c < C; ++c)
    if (m->calls[c].sample_end.empty()) return kfail(PSATTN_E_INVALID_ARG, "call %d has no sample", c);
  // next use of each node after call c: for eviction (farthest next use first)
  const int kNever = std::numeric_limits<int>::max();
  auto next_use = [&](int n, int c) {
    for (int k = c + 1; k < C; ++k)
      if (reads[k][n]) return k;
    return kNever;
  };

  SlotAllocator pool(m->capacity);
  std::vector<std::vector<Page>> live(N);   // current blocks of each cached node
  std::vector<char> computed(N, 0);
  const int32_t B = o.block_size;
  auto pages_of = [&](int n) {
    std::vector<Page> p;
    if (B <= 0) {
      p.push_back({0, seg_len[n], seg_len[n]});
    } else {
      for (int32_t k = 0; k < seg_len[n]; k += B) p.push_back({0, B, std::min(B, seg_len[n] - k)});
    }
    return p;
  };
  auto release = [&](int n) {
    for (const Page& pg : live[n]) pool.release(pg.base, pg.cap);
    live[n].clear();
  };
  int64_t peak = 0;
  for (int c = 0; c < C; ++c) {
    CallPlan& cp = m->calls[c];
    for (int n = 0; n < N; ++n)
      if (reads[c][n]) cp.nodes.push_back(n);
    std::vector<char> need(N, 0);
    for (int n : cp.nodes) need[n] = 1;
    for (int n : cp.nodes) {
      const bool cached = !live[n].empty();
      cp.ext.push_back(computed[n] ? 1 : 0);
      if (cached) {
        cp.pages.push_back(live[n]);
        continue;
      }
      std::vector<Page> pg = pages_of(n);
      for (Page& p : pg) {
        while (!pool.alloc(p.cap, &p.base)) {
          // evict the cached block the call does not need with the farthest next use
          int victim = -1, vuse = -1;
          for (int v = 0; v < N; ++v) {
            if (live[v].empty() || need[v]) continue;
            const int u = next_use(v, c);
            if (u > vuse) {
              vuse = u;
              victim = v;
            }
          }
          if (victim < 0)
            return kfail(PSATTN_E_WORKSPACE,
                         "call %d: node %d needs %d more slots; the pool of %lld holds %lld in blocks this call reads",
                         c, n, p.cap, (long long)m->capacity, (long long)pool.used());
          cp.before.push_back(event(PSATTN_KVM_EVICT, victim, live[victim]));
          m->stats.evictions += 1;
          release(victim);
        }
      }
      live[n] = pg;
      cp.pages.push_back(pg);
      cp.before.push_back(event(computed[n] ? PSATTN_KVM_REFILL : PSATTN_KVM_ALLOC, n, pg));
      if (computed[n]) m->stats.refilled_tokens += seg_len[n];
      m->stats.allocated_tokens += seg_len[n];
    }
    for (int n : cp.nodes) computed[n] = 1;
    cp.used = pool.used();
    peak = std::max(peak, cp.used);
    // after the call's backward: reference counts (Sec. 5.2)
    for (int n : cp.nodes) {
      refcount[n] -= reads[c][n];
      const bool last = c == C - 1;
      if ((o.dbc && refcount[n] == 0) || (!o.dbc && last)) {
        cp.after.push_back(event(PSATTN_KVM_FREE, n, live[n]));
        release(n);
      }
    }
    if (!o.dbc && c == C - 1)   // everything else cached is dropped at the end of the schedule
      for (int n = 0; n < N; ++n)
        if (!live[n].empty()) {
          cp.after.push_back(event(PSATTN_KVM_FREE, n, live[n]));
          release(n);
        }
  }
  m->stats.peak_slots = peak;
  m->stats.final_slots = pool.used();
  m->stats.num_calls = C;

  // descriptors
  for (int c = 0; c < C; ++c) {
    CallPlan& cp = m->calls[c];
    std::vector<int32_t> local(N, -1);
    for (size_t i = 0; i < cp.nodes.size(); ++i) local[cp.nodes[i]] = (int32_t)i;
    int64_t row = 0;
    cp.d_blk_ptr.push_back(0);
    for (size_t i = 0; i < cp.nodes.size(); ++i) {
      const int n = cp.nodes[i];
      cp.d_parent.push_back(parent[n] < 0 ? -1 : local[parent[n]]);
      cp.d_seg.push_back(seg_len[n]);
      cp.d_row_off.push_back(cp.ext[i] ? -1 : row);
      if (!cp.ext[i]) row += seg_len[n];
      int64_t pos = off[n];
      for (const Page& p : cp.pages[i]) {
        cp.d_blocks.push_back({p.base, p.cap, p.len, (int32_t)pos, 0});
        pos += p.len;
      }
      cp.d_blk_ptr.push_back((int32_t)cp.d_blocks.size());
    }
    for (int32_t e : cp.sample_end) cp.d_end.push_back(local[e]);
  }
  return PSATTN_OK;
}

}  // namespace

extern "C" psattn_status psattn_kvm_plan(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                                         int32_t num_samples, const int32_t* sample_end, const int32_t* call_of_sample,
                                         const psattn_kvm_opts* opts, psattn_kvm** out) {
  if (!out) return kfail(PSATTN_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (num_nodes < 1 || num_samples < 1 || !parent || !seg_len || !sample_end || !call_of_sample || !opts)
    return kfail(PSATTN_E_INVALID_ARG, "need num_nodes, num_samples >= 1 and non-NULL arrays and options");
  for (int i = 0; i < 4; ++i)
    if (opts->reserved[i]) return kfail(PSATTN_E_INVALID_ARG, "psattn_kvm_opts.reserved must be zero");
  if (opts->capacity_slots < 1) return kfail(PSATTN_E_INVALID_ARG, "capacity_slots must be >= 1");
  if (opts->block_size < 0) return kfail(PSATTN_E_INVALID_ARG, "block_size must be >= 0");
  psattn_kvm* m = new (std::nothrow) psattn_kvm;
  if (!m) return kfail(PSATTN_E_INVALID_ARG, "out of host memory");
  m->N = num_nodes;
  m->S = num_samples;
  m->capacity = opts->capacity_slots;
  psattn_status st;
  try {
    st = build(m, parent, seg_len, sample_end, call_of_sample, *opts);
  } catch (const std::bad_alloc&) {
    st = kfail(PSATTN_E_INVALID_ARG, "out of host memory");
  }
  if (st != PSATTN_OK) {
    delete m;
    return st;
  }
  *out = m;
  return PSATTN_OK;
}

extern "C" void psattn_kvm_destroy(psattn_kvm* m) { delete m; }

extern "C" psattn_status psattn_kvm_call_desc(const psattn_kvm* m, int32_t call, psattn_tree_desc* desc,
                                              const int32_t** node_ids) {
  if (!m || !desc) return kfail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (call < 0 || call >= m->C) return kfail(PSATTN_E_INVALID_ARG, "call %d out of range [0, %d)", call, m->C);
  const CallPlan& cp = m->calls[call];
  desc->num_nodes = (int32_t)cp.nodes.size();
  desc->parent = cp.d_parent.data();
  desc->seg_len = cp.d_seg.data();
  desc->row_off = cp.d_row_off.data();
  desc->blk_ptr = cp.d_blk_ptr.data();
  desc->blocks = cp.d_blocks.data();
  desc->pool_slots = m->capacity;
  desc->num_samples = (int32_t)cp.d_end.size();
  desc->sample_end = cp.d_end.data();
  if (node_ids) *node_ids = cp.nodes.data();
  return PSATTN_OK;
}

extern "C" psattn_status psattn_kvm_events(const psattn_kvm* m, int32_t call, int32_t phase,
                                           const psattn_kvm_event** events, int32_t* count) {
  if (!m || !events || !count) return kfail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (call < 0 || call >= m->C) return kfail(PSATTN_E_INVALID_ARG, "call %d out of range [0, %d)", call, m->C);
  if (phase != 0 && phase != 1) return kfail(PSATTN_E_INVALID_ARG, "phase must be 0 (before) or 1 (after)");
  const std::vector<psattn_kvm_event>& v = phase ? m->calls[call].after : m->calls[call].before;
  *events = v.data();
  *count = (int32_t)v.size();
  return PSATTN_OK;
}

extern "C" psattn_status psattn_kvm_get_stats(const psattn_kvm* m, psattn_kvm_stats* stats, int64_t* used_per_call) {
  if (!m || !stats) return kfail(PSATTN_E_INVALID_ARG, "NULL argument");
  *stats = m->stats;
  if (used_per_call)
    for (int c = 0; c < m->C; ++c) used_per_call[c] = m->calls[c].used;
  return PSATTN_OK;
}
