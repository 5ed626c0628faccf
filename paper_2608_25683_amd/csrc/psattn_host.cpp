// Host side of the prefix-shared attention library: descriptor validation,
// the tree-to-tile planner, plan upload, workspace sizing, launch sequencing
// and kernel timing.  Implements the C ABI declared in include/psattn.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <numeric>
#include <string>
#include <vector>

#include "psattn.h"
#include "psattn_launch.h"
#include "psattn_plan.h"

using namespace psattn;

namespace {

thread_local std::string g_err;

psattn_status fail(psattn_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

}  // namespace

namespace psattn {
// the thread-local last-error message, for the library's other sources
psattn_status set_error(psattn_status st, const char* msg) { return fail(st, "%s", msg); }
}  // namespace psattn

struct psattn_tree {
  // descriptor (copied)
  int32_t N = 0, S = 0, hq = 0, hkv = 0, d = 0;
  float scale = 0.f;
  psattn_dtype dtype = PSATTN_BF16;
  int64_t pool_slots = 0;
  std::vector<int32_t> parent, seg_len, blk_ptr, sample_end;
  std::vector<int64_t> row_off;
  std::vector<psattn_block> blocks;
  // derived tree facts
  std::vector<int64_t> off;        // sequence position of each node's first token
  std::vector<char> ext;           // node cached by an earlier call: K/V in the pool, no query rows here
  std::vector<int32_t> refcount;   // samples whose path holds the node (Sec. 5.2)
  std::vector<std::vector<int32_t>> children;
  int64_t Ns = 0, Nu = 0, nvis = 0;
  // plan (host copy)
  Shape shape{};
  std::vector<int32_t> row_pos, row_slot, q_list, q_pos, kv_list, pad_slots;
  std::vector<FwdItem> fwd;
  std::vector<MergeEntry> merge;
  std::vector<BkvItem> bkv;
  std::vector<ReduceEntry> reduce;
  int64_t fwd_part_rows = 0, bkv_part_tiles = 0;
  // device image of the plan
  size_t o_row_pos = 0, o_row_slot = 0, o_q = 0, o_qpos = 0, o_kv = 0, o_fwd = 0, o_merge = 0, o_bkv = 0, o_reduce = 0, o_pad = 0;
  size_t plan_bytes = 0;
  std::vector<uint8_t> image;
  void* dev = nullptr;
  size_t dev_bytes = 0;
};

namespace {

// --------------------------------------------------------------------------------------------
// Validation (descriptor ingest)

psattn_status validate_and_copy(const psattn_tree_desc* d, psattn_tree* t) {
  if (!d) return fail(PSATTN_E_INVALID_ARG, "desc is NULL");
  if (d->num_nodes < 1) return fail(PSATTN_E_INVALID_ARG, "num_nodes must be >= 1 (got %d)", d->num_nodes);
  if (d->num_samples < 1) return fail(PSATTN_E_INVALID_ARG, "num_samples must be >= 1 (got %d)", d->num_samples);
  if (!d->parent || !d->seg_len || !d->row_off || !d->blk_ptr || !d->blocks || !d->sample_end)
    return fail(PSATTN_E_INVALID_ARG, "a descriptor array pointer is NULL");
  if (d->hq < 1 || d->hkv < 1 || d->hq % d->hkv != 0)
    return fail(PSATTN_E_UNSUPPORTED, "hq (%d) must be a positive multiple of hkv (%d)", d->hq, d->hkv);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(PSATTN_E_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", d->head_dim);
  if (d->dtype != PSATTN_BF16 && d->dtype != PSATTN_FP32)
    return fail(PSATTN_E_UNSUPPORTED, "unknown dtype %d", (int)d->dtype);
  if (!(d->softmax_scale > 0.f) || !std::isfinite(d->softmax_scale))
    return fail(PSATTN_E_INVALID_ARG, "softmax_scale must be positive and finite");
  if (d->pool_slots < 1 || d->pool_slots > INT32_MAX)
    return fail(PSATTN_E_UNSUPPORTED, "pool_slots must be in [1, 2^31) (got %lld)", (long long)d->pool_slots);

  const int N = d->num_nodes;
  t->N = N;
  t->S = d->num_samples;
  t->hq = d->hq;
  t->hkv = d->hkv;
  t->d = d->head_dim;
  t->scale = d->softmax_scale;
  t->dtype = d->dtype;
  t->pool_slots = d->pool_slots;
  t->parent.assign(d->parent, d->parent + N);
  t->seg_len.assign(d->seg_len, d->seg_len + N);
  t->row_off.assign(d->row_off, d->row_off + N);
  t->blk_ptr.assign(d->blk_ptr, d->blk_ptr + N + 1);
  t->sample_end.assign(d->sample_end, d->sample_end + t->S);

  // parents precede children; segments non-empty; external (cached) nodes only above external
  // nodes, so that they form a prefix of every path that holds them (Sec. 4.1.1, 4.1.2)
  t->off.assign(N, 0);
  t->ext.assign(N, 0);
  t->children.assign(N, {});
  int64_t ns = 0;
  for (int i = 0; i < N; ++i) {
    int p = t->parent[i];
    if (p < -1 || p >= i)
      return fail(PSATTN_E_INVALID_TREE, "parent[%d] = %d: a parent must precede its child (or be -1)", i, p);
    if (t->seg_len[i] < 1) return fail(PSATTN_E_INVALID_TREE, "seg_len[%d] = %d: segments must be non-empty", i, t->seg_len[i]);
    t->ext[i] = t->row_off[i] < 0;
    if (t->ext[i] && p >= 0 && !t->ext[p])
      return fail(PSATTN_E_INVALID_TREE, "node %d is external (row_off < 0) but its parent %d is not", i, p);
    t->off[i] = p < 0 ? 0 : t->off[p] + t->seg_len[p];
    if (p >= 0) t->children[p].push_back(i);
    if (!t->ext[i]) ns += t->seg_len[i];
    if (t->off[i] + t->seg_len[i] > INT32_MAX) return fail(PSATTN_E_UNSUPPORTED, "sequence of node %d too long", i);
  }
  if (ns < 1) return fail(PSATTN_E_INVALID_TREE, "every node is external: the call has no query rows");
  if (ns > INT32_MAX / 2) return fail(PSATTN_E_UNSUPPORTED, "too many rows (%lld)", (long long)ns);
  t->Ns = ns;
  if (t->dtype == PSATTN_BF16) {
    // the bf16 kernels address the K/V pools and the Q / O / dO tensors by 32-bit byte offsets
    // and pool slots by 24-bit products
    const int64_t kv_bytes = t->pool_slots * t->hkv * t->d * 2, q_bytes = ns * t->hq * t->d * 2;
    if (t->pool_slots > (1 << 24) || kv_bytes > (int64_t)UINT32_MAX)
      return fail(PSATTN_E_UNSUPPORTED, "bf16 pool of %lld slots (%lld bytes per tensor): at most 2^24 slots and 4 GiB",
                  (long long)t->pool_slots, (long long)kv_bytes);
    if (q_bytes > (int64_t)UINT32_MAX || ns * t->hq >= (1 << 24))
      return fail(PSATTN_E_UNSUPPORTED, "bf16 query tensor of %lld rows x %d heads: at most 4 GiB and 2^24 row-heads",
                  (long long)ns, t->hq);
  }

  // row ranges of the internal nodes tile [0, Ns)
  {
    std::vector<int> ord;
    for (int i = 0; i < N; ++i)
      if (!t->ext[i]) ord.push_back(i);
    std::sort(ord.begin(), ord.end(), [&](int a, int b) { return t->row_off[a] < t->row_off[b]; });
    int64_t cur = 0;
    for (size_t k = 0; k < ord.size(); ++k) {
      int i = ord[k];
      if (t->row_off[i] != cur)
        return fail(PSATTN_E_INVALID_TREE, "row_off[%d] = %lld: node row ranges must tile [0, Ns) without gaps or overlap",
                    i, (long long)t->row_off[i]);
      cur += t->seg_len[i];
    }
  }

  // blocks
  if (t->blk_ptr[0] != 0) return fail(PSATTN_E_INVALID_ARG, "blk_ptr[0] must be 0");
  for (int i = 0; i < N; ++i)
    if (t->blk_ptr[i + 1] <= t->blk_ptr[i])
      return fail(PSATTN_E_BLOCK_COVERAGE, "node %d owns no block (blk_ptr must increase)", i);
  const int nb = t->blk_ptr[N];
  t->blocks.assign(d->blocks, d->blocks + nb);
  for (int i = 0; i < N; ++i) {
    int64_t pos = t->off[i];
    int64_t tot = 0;
    for (int b = t->blk_ptr[i]; b < t->blk_ptr[i + 1]; ++b) {
      const psattn_block& B = t->blocks[b];
      if (B.capacity < 1 || B.len < 1 || B.len > B.capacity)
        return fail(PSATTN_E_BLOCK_RANGE, "block %d: need 1 <= len (%d) <= capacity (%d)", b, B.len, B.capacity);
      if (B.base < 0 || B.base + B.capacity > t->pool_slots)
        return fail(PSATTN_E_BLOCK_RANGE, "block %d: slots [%lld, %lld) outside the pool of %lld", b, (long long)B.base,
                    (long long)(B.base + B.capacity), (long long)t->pool_slots);
      if (B.pos != pos)
        return fail(PSATTN_E_BLOCK_COVERAGE, "block %d: pos %d, expected %lld (node %d offset + earlier blocks)", b, B.pos,
                    (long long)pos, i);
      pos += B.len;
      tot += B.len;
    }
    if (tot != t->seg_len[i])
      return fail(PSATTN_E_BLOCK_COVERAGE, "node %d: blocks hold %lld tokens, segment has %d", i, (long long)tot, t->seg_len[i]);
  }
  {
    std::vector<int> ord(nb);
    std::iota(ord.begin(), ord.end(), 0);
    std::sort(ord.begin(), ord.end(), [&](int a, int b) { return t->blocks[a].base < t->blocks[b].base; });
    for (int k = 1; k < nb; ++k) {
      const psattn_block& A = t->blocks[ord[k - 1]];
      const psattn_block& B = t->blocks[ord[k]];
      if (B.base < A.base + A.capacity)
        return fail(PSATTN_E_BLOCK_OVERLAP, "blocks %d and %d overlap in the pool", ord[k - 1], ord[k]);
    }
  }

  // samples and reference counts (Sec. 5.2: samples that will read each block)
  t->refcount.assign(N, 0);
  int64_t nu = 0;
  for (int s = 0; s < t->S; ++s) {
    int e = t->sample_end[s];
    if (e < 0 || e >= N) return fail(PSATTN_E_INVALID_TREE, "sample_end[%d] = %d out of range", s, e);
    if (t->ext[e]) return fail(PSATTN_E_INVALID_TREE, "sample_end[%d] = %d is an external node (no query rows here)", s, e);
    for (int n = e; n >= 0; n = t->parent[n]) {
      t->refcount[n]++;
      if (!t->ext[n]) nu += t->seg_len[n];   // unshared-equivalent query tokens of this call
    }
  }
  t->Nu = nu;
  for (int i = 0; i < N; ++i) {
    if (t->refcount[i] == 0)
      return fail(PSATTN_E_INVALID_TREE, "node %d lies on no sample path (its outputs would be undefined)", i);
    for (int b = t->blk_ptr[i]; b < t->blk_ptr[i + 1]; ++b)
      if (t->blocks[b].refcount != 0 && t->blocks[b].refcount != t->refcount[i])
        return fail(PSATTN_E_INVALID_TREE, "block %d: refcount %d, but %d samples read node %d", b, t->blocks[b].refcount,
                    t->refcount[i], i);
  }
  int64_t nvis = 0;
  for (int i = 0; i < N; ++i) {
    if (t->ext[i]) continue;
    int64_t L = t->seg_len[i];
    nvis += L * t->off[i] + L * (L + 1) / 2;
  }
  t->nvis = nvis;
  return PSATTN_OK;
}

// --------------------------------------------------------------------------------------------
// Planner

struct Task {
  double cost;
  int idx;
};

// Longest-first order (the greedy placement of Sec. 4.2 applied to work items:
// the hardware dispatcher hands the next item to whichever compute unit frees first).
std::vector<int> longest_first(const std::vector<double>& cost) {
  std::vector<int> ord(cost.size());
  std::iota(ord.begin(), ord.end(), 0);
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return cost[a] > cost[b]; });
  return ord;
}

#ifdef PSATTN_PLAN_CHECKS
// Opt-in (-DPSATTN_PLAN_CHECKS): every index the kernels derive from the plan lies inside the
// array or buffer it addresses -- row and slot lists, item ranges, partial rows and tiles.  The
// sanitized host build of the tests compiles it in.
psattn_status check_plan(const psattn_tree* t) {
  const int64_t nql = (int64_t)t->q_list.size(), nkl = (int64_t)t->kv_list.size();
  const int64_t ns = t->shape.ns, slots = t->pool_slots;
  auto bad = [&](const char* what, int64_t i) {
    return fail(PSATTN_E_INTERNAL, "plan check: %s (entry %lld)", what, (long long)i);
  };
  for (int64_t i = 0; i < ns; ++i) {
    if (t->row_pos[i] < 0) return bad("row position < 0", i);
    if (t->row_slot[i] < 0 || t->row_slot[i] >= slots) return bad("row slot outside the pool", i);
  }
  for (int64_t i = 0; i < nql; ++i)
    if (t->q_list[i] < 0 || t->q_list[i] >= ns) return bad("q_list row outside [0, Ns)", i);
  if ((int64_t)t->q_pos.size() != nql) return bad("q_pos length", (int64_t)t->q_pos.size());
  for (int64_t i = 0; i < nql; ++i)
    if (t->q_pos[i] != t->row_pos[t->q_list[i]]) return bad("q_pos entry", i);
  for (int64_t i = 0; i < nkl; ++i)
    if (t->kv_list[i] < 0 || t->kv_list[i] >= slots) return bad("kv_list slot outside the pool", i);
  for (size_t i = 0; i < t->pad_slots.size(); ++i)
    if (t->pad_slots[i] < 0 || t->pad_slots[i] >= slots) return bad("pad slot outside the pool", (int64_t)i);
  const Shape& s = t->shape;
  for (size_t i = 0; i < t->fwd.size(); ++i) {
    const FwdItem& f = t->fwd[i];
    if (f.nq < 1 || f.nq > s.bmq || f.q_off < 0 || (int64_t)f.q_off + f.nq > nql) return bad("forward item rows", (int64_t)i);
    if (f.nkv < 1 || f.kv_off < 0 || (int64_t)f.kv_off + f.nkv > nkl) return bad("forward item keys", (int64_t)i);
    if (f.head0 < 0 || f.head0 + s.hc > s.hq || f.head0 / s.g != (f.head0 + s.hc - 1) / s.g) return bad("forward item heads", (int64_t)i);
    if (f.part < -1 || (f.part >= 0 && (int64_t)f.part + f.nq > t->fwd_part_rows)) return bad("forward item partial rows", (int64_t)i);
    if (f.nfull < 0 || (int64_t)f.nfull * KV_TILE > f.nkv + KV_TILE - 1) return bad("forward item unmasked tiles", (int64_t)i);
  }
  for (size_t i = 0; i < t->merge.size(); ++i) {
    const MergeEntry& m = t->merge[i];
    if (m.nq < 1 || m.q_off < 0 || (int64_t)m.q_off + m.nq > nql) return bad("merge rows", (int64_t)i);
    if (m.nparts < 1 || m.part0 < 0 || (int64_t)m.part0 + (int64_t)(m.nparts - 1) * s.bmq + m.nq > t->fwd_part_rows)
      return bad("merge partial rows", (int64_t)i);
  }
  for (size_t i = 0; i < t->bkv.size(); ++i) {
    const BkvItem& b = t->bkv[i];
    if (b.nk < 1 || b.nk > BKV_TILE || b.kv_off < 0 || (int64_t)b.kv_off + b.nk > nkl) return bad("dK/dV item keys", (int64_t)i);
    if (b.nq < 1 || b.q_off < 0 || (int64_t)b.q_off + b.nq > nql) return bad("dK/dV item rows", (int64_t)i);
    if (b.hk < 0 || b.hk >= s.hkv) return bad("dK/dV item kv head", (int64_t)i);
    if (b.part < -1 || b.part >= t->bkv_part_tiles) return bad("dK/dV item partial tile", (int64_t)i);
    if (b.mask_lo < 0 || b.mask_lo > b.mask_hi || b.mask_hi > b.nq) return bad("dK/dV item mask range", (int64_t)i);
  }
  for (size_t i = 0; i < t->reduce.size(); ++i) {
    const ReduceEntry& r = t->reduce[i];
    if (r.nk < 1 || r.nk > BKV_TILE || r.kv_off < 0 || (int64_t)r.kv_off + r.nk > nkl) return bad("reduce keys", (int64_t)i);
    if (r.hk < 0 || r.hk >= s.hkv) return bad("reduce kv head", (int64_t)i);
    if (r.nparts < 1 || r.part0 < 0 || (int64_t)r.part0 + r.nparts > t->bkv_part_tiles) return bad("reduce partial tiles", (int64_t)i);
  }
  return PSATTN_OK;
}
#endif

psattn_status build_plan(psattn_tree* t, const psattn_plan_opts& o) {
  const int N = t->N;
  Shape& s = t->shape;
  s.ns = (int32_t)t->Ns;
  s.hq = t->hq;
  s.hkv = t->hkv;
  s.d = t->d;
  s.g = t->hq / t->hkv;
  // Heads per forward/dQ item: the largest common divisor of G and 4, and 32-row subtiles per
  // head rw = 8 / hc (2, 4 or 8).  Every item is then 8 subtile x head pairs, which the
  // eight-wavefront kernels need, and each staged key tile serves 8 x 32 query-head rows.  (For
  // G = 5 or 7 that means one head per item with 256-row query tiles.)
  s.hc = s.g % 4 == 0 ? 4 : (s.g % 2 == 0 ? 2 : 1);
  s.rw = 8 / s.hc;
  s.nw = s.hc * s.rw;
  s.bmq = Q_SUB * s.rw;
  s.scale = t->scale;
  const int n_chunks = t->hq / s.hc;  // head chunks per forward task
  const int num_cus = o.num_cus > 0 ? o.num_cus : 256;

  // pool slots of every node's tokens, and sequence position of every packed row
  std::vector<std::vector<int32_t>> node_slots(N);
  t->row_pos.assign(t->Ns, 0);
  t->row_slot.assign(t->Ns, 0);
  for (int n = 0; n < N; ++n) {
    for (int b = t->blk_ptr[n]; b < t->blk_ptr[n + 1]; ++b)
      for (int k = 0; k < t->blocks[b].len; ++k) node_slots[n].push_back((int32_t)(t->blocks[b].base + k));
    if (!t->ext[n])
      for (int a = 0; a < t->seg_len[n]; ++a) {
        t->row_pos[t->row_off[n] + a] = (int32_t)(t->off[n] + a);
        t->row_slot[t->row_off[n] + a] = node_slots[n][a];
      }
  }

  // per-node path slot list: slots of sequence positions 0 .. off+len-1
  std::vector<int64_t> kvoff(N);
  t->kv_list.clear();
  for (int n = 0; n < N; ++n) {
    std::vector<int> path;
    for (int m = n; m >= 0; m = t->parent[m]) path.push_back(m);
    std::reverse(path.begin(), path.end());
    kvoff[n] = (int64_t)t->kv_list.size();
    for (int m : path) t->kv_list.insert(t->kv_list.end(), node_slots[m].begin(), node_slots[m].end());
    if (t->kv_list.size() > (size_t)INT32_MAX) return fail(PSATTN_E_UNSUPPORTED, "key lists exceed 2^31 entries");
  }

  // ---------------- forward / dQ tasks: query tile x key range (pieces) ----------------
  struct FTask { int32_t q_off, nq, kv_off, kv_pos0, nkv, min_qpos, part; double cost; };
  std::vector<FTask> ftasks;
  std::vector<MergeEntry> merges;
  t->q_list.clear();
  int64_t total_f = 0;
  for (int n = 0; n < N; ++n)
    for (int a0 = 0; !t->ext[n] && a0 < t->seg_len[n]; a0 += s.bmq) {
      int a1 = std::min<int>(t->seg_len[n], a0 + s.bmq);
      total_f += (int64_t)(a1 - a0) * (t->off[n] + a1);
    }
  int64_t split_keys;
  if (o.fwd_kv_split > 0) {
    split_keys = ((int64_t)o.fwd_kv_split + KV_TILE - 1) / KV_TILE * KV_TILE;
  } else if (o.fwd_kv_split < 0) {
    split_keys = INT64_MAX;
  } else {
    // automatic: split only when a single item would dominate an even share of the work
    int64_t per_cu = total_f * n_chunks / std::max(1, 2 * num_cus);
    split_keys = std::max<int64_t>(16 * KV_TILE, per_cu / std::max(1, s.bmq) / KV_TILE * KV_TILE);
  }
  int64_t part_rows = 0;
  // Sibling packing: children of one parent whose segments fill at most half a query tile share
  // the key range [0, off) of their common prefix.  Their rows are packed (first fit, child
  // order) into one tile for that range, and each node keeps an item of its own keys
  // [off, off + seg).  A pack's partial rows: prefix piece j of the node at pack offset o at
  // P + j*bmq + o, the node's own piece at P + npref*bmq + o, so that one merge record per node
  // (part0 = P + o, npref + 1 parts) combines them.
  std::vector<char> packed(N, 0);
  std::vector<std::vector<int>> packs;
  for (int p = 0; p < N; ++p) {
    std::vector<int> cur;
    int rows = 0;
    auto flush = [&]() {
      if (cur.size() >= 2) {
        for (int c : cur) packed[c] = 1;
        packs.push_back(cur);
      }
      cur.clear();
      rows = 0;
    };
    for (int c : t->children[p]) {
      if (t->ext[c] || 2 * t->seg_len[c] > s.bmq) continue;
      if (rows + t->seg_len[c] > s.bmq) flush();
      cur.push_back(c);
      rows += t->seg_len[c];
    }
    flush();
  }
  auto split_range = [&](int64_t nkv_total) {
    return split_keys == INT64_MAX ? 1 : (int)((nkv_total + split_keys - 1) / split_keys);
  };
  for (const std::vector<int>& pk : packs) {
    const int n0 = pk[0];
    const int64_t pre = t->off[n0];   // the common prefix: every sibling starts at the same position
    const int npref = split_range(pre);
    const int32_t P = (int32_t)part_rows;
    part_rows += (int64_t)(npref + 1) * s.bmq;
    const int32_t q_pack = (int32_t)t->q_list.size();
    int rows = 0;
    for (int n : pk)
      for (int a = 0; a < t->seg_len[n]; ++a) t->q_list.push_back((int32_t)(t->row_off[n] + a));
    for (int j = 0; j < npref; ++j) {
      const int64_t k0 = npref > 1 ? j * split_keys : 0;
      const int64_t k1 = npref > 1 ? std::min(pre, (j + 1) * split_keys) : pre;
      FTask f;
      f.q_off = q_pack;
      f.nq = (int32_t)(t->q_list.size() - q_pack);
      f.kv_off = (int32_t)(kvoff[n0] + k0);
      f.kv_pos0 = (int32_t)k0;
      f.nkv = (int32_t)(k1 - k0);
      f.min_qpos = (int32_t)pre;
      f.part = P + j * s.bmq;
      f.cost = (double)f.nq * (double)f.nkv + 4096.0;
      ftasks.push_back(f);
    }
    for (int n : pk) {
      const int32_t q_off = (int32_t)t->q_list.size();
      for (int a = 0; a < t->seg_len[n]; ++a) t->q_list.push_back((int32_t)(t->row_off[n] + a));
      merges.push_back({q_off, t->seg_len[n], P + rows, npref + 1});
      FTask f;
      f.q_off = q_off;
      f.nq = t->seg_len[n];
      f.kv_off = (int32_t)(kvoff[n] + pre);
      f.kv_pos0 = (int32_t)pre;
      f.nkv = t->seg_len[n];
      f.min_qpos = (int32_t)pre;
      f.part = P + npref * s.bmq + rows;
      f.cost = (double)f.nq * (double)f.nkv + 4096.0;
      ftasks.push_back(f);
      rows += t->seg_len[n];
    }
  }
  for (int n = 0; n < N; ++n) {
    if (packed[n] || t->ext[n]) continue;
    for (int a0 = 0; a0 < t->seg_len[n]; a0 += s.bmq) {
      int a1 = std::min<int>(t->seg_len[n], a0 + s.bmq);
      int nq = a1 - a0;
      int32_t q_off = (int32_t)t->q_list.size();
      for (int a = a0; a < a1; ++a) t->q_list.push_back((int32_t)(t->row_off[n] + a));
      int64_t nkv_total = t->off[n] + a1;
      int64_t min_qpos = t->off[n] + a0;
      const int npieces = split_keys == INT64_MAX ? 1 : (int)((nkv_total + split_keys - 1) / split_keys);
      int32_t part0 = -1;
      if (npieces > 1) {
        part0 = (int32_t)part_rows;
        part_rows += (int64_t)npieces * s.bmq;
        merges.push_back({q_off, nq, part0, npieces});
      }
      for (int j = 0; j < npieces; ++j) {
        int64_t k0 = npieces > 1 ? j * split_keys : 0;
        int64_t k1 = npieces > 1 ? std::min(nkv_total, (j + 1) * split_keys) : nkv_total;
        FTask f;
        f.q_off = q_off;
        f.nq = nq;
        f.kv_off = (int32_t)(kvoff[n] + k0);
        f.kv_pos0 = (int32_t)k0;
        f.nkv = (int32_t)(k1 - k0);
        f.min_qpos = (int32_t)min_qpos;
        f.part = npieces > 1 ? part0 + j * s.bmq : -1;
        f.cost = (double)nq * (double)f.nkv + 4096.0;  // Eq. "single_sequence": alpha1 * l_suf * l + alpha3
        ftasks.push_back(f);
      }
    }
  }
  if (part_rows > INT32_MAX / 2) return fail(PSATTN_E_UNSUPPORTED, "too many partial rows");
  t->fwd_part_rows = part_rows;
  t->merge = merges;
  {
    std::vector<double> c(ftasks.size());
    for (size_t i = 0; i < ftasks.size(); ++i) c[i] = ftasks[i].cost;
    t->fwd.clear();
    for (int i : longest_first(c)) {
      const FTask& f = ftasks[i];
      int64_t full_by_len = f.nkv / KV_TILE;
      int64_t full_by_mask = (int64_t)f.min_qpos + 1 - f.kv_pos0;
      full_by_mask = full_by_mask < 0 ? 0 : full_by_mask / KV_TILE;
      int32_t nfull = (int32_t)std::min(full_by_len, full_by_mask);
      // the task's head chunks with the kv head varying fastest: consecutive workgroups, which the
      // dispatcher deals round-robin to the 8 XCDs, then read one kv head per XCD (each XCD's L2
      // holds one kv head's K/V) whatever the number of query heads per kv head
      for (int j = 0; j < n_chunks; ++j) {
        const int kvh = j % t->hkv, sub = j / t->hkv;
        t->fwd.push_back({f.q_off, f.nq, f.kv_off, f.nkv, f.kv_pos0, kvh * s.g + sub * s.hc, f.part, nfull});
      }
    }
  }

  // ---------------- dK/dV tasks: key tile x consumer-row chunk ----------------
  // consumer list of node m: every row of every (internal) descendant (node order), then m's own
  // rows from its last position down to 0; the tile starting at key b0 uses the list up to own
  // position b0.  An external node has no own rows: all its consumers see every key of a tile.
  std::vector<int64_t> cons_off(N), cons_len(N), desc_len(N);
  for (int m = 0; m < N; ++m) {
    cons_off[m] = (int64_t)t->q_list.size();
    std::vector<int> stack(t->children[m].begin(), t->children[m].end());
    std::vector<int> sub;
    while (!stack.empty()) {
      int x = stack.back();
      stack.pop_back();
      sub.push_back(x);
      for (int c : t->children[x]) stack.push_back(c);
    }
    std::sort(sub.begin(), sub.end());
    for (int x : sub)
      for (int a = 0; !t->ext[x] && a < t->seg_len[x]; ++a) t->q_list.push_back((int32_t)(t->row_off[x] + a));
    desc_len[m] = (int64_t)t->q_list.size() - cons_off[m];
    for (int a = t->seg_len[m] - 1; !t->ext[m] && a >= 0; --a) t->q_list.push_back((int32_t)(t->row_off[m] + a));
    cons_len[m] = (int64_t)t->q_list.size() - cons_off[m];
    if (t->q_list.size() > (size_t)INT32_MAX) return fail(PSATTN_E_UNSUPPORTED, "row lists exceed 2^31 entries");
  }
  int64_t total_b = 0;
  for (int m = 0; m < N; ++m)
    for (int b0 = 0; b0 < t->seg_len[m]; b0 += BKV_TILE) {
      int nk = std::min(BKV_TILE, t->seg_len[m] - b0);
      total_b += (int64_t)nk * (cons_len[m] - (t->ext[m] ? 0 : b0));
    }
  int64_t chunk_rows;
  if (o.bwd_q_chunk > 0) {
    chunk_rows = ((int64_t)o.bwd_q_chunk + Q_SUB - 1) / Q_SUB * Q_SUB;
  } else if (o.bwd_q_chunk < 0) {
    chunk_rows = INT64_MAX;
  } else {
    // a chunk holds at most one CU's share of the dK/dV work: a tile whose consumers fit in one
    // share runs as one item, with no partial tiles to write and sum
    int64_t per_cu = total_b * t->hkv / std::max(1, num_cus);
    chunk_rows = std::max<int64_t>(2048, per_cu / BKV_TILE / Q_SUB * Q_SUB);
  }
  struct BTask {
    int32_t kv_off, nk, kv_pos0, q_off, nq, mask_lo, mask_hi, part_base, nparts, chunk, acc;
    double cost, key;
    int64_t group;   // tasks of one group (same key and group) are emitted as one run
  };
  std::vector<BTask> btasks;
  std::vector<ReduceEntry> reduces;
  int64_t part_tiles = 0;
  for (int m = 0; m < N; ++m) {
    const size_t first_task = btasks.size();
    for (int b0 = 0; b0 < t->seg_len[m]; b0 += BKV_TILE) {
      int nk = std::min(BKV_TILE, t->seg_len[m] - b0);
      // an external node's tiles add this call's consumers to the gradients that earlier calls
      // left in dK/dV (the cached block's accumulators)
      const int acc = t->ext[m] ? 1 : 0;
      int64_t nq_total = cons_len[m] - (acc ? 0 : b0);
      // own rows at positions b0 .. b0+nk-2 see only part of the tile: the last nk-1 list entries
      const int64_t mlo = acc ? nq_total : nq_total - (nk - 1), mhi = nq_total;
      int nparts = chunk_rows == INT64_MAX ? 1 : (int)((nq_total + chunk_rows - 1) / chunk_rows);
      int32_t kv_off = (int32_t)(kvoff[m] + t->off[m] + b0);
      int32_t kv_pos0 = (int32_t)(t->off[m] + b0);
      int32_t part_base = -1;
      if (nparts > 1) {
        part_base = (int32_t)part_tiles;
        part_tiles += (int64_t)nparts * t->hkv;
        for (int hk = 0; hk < t->hkv; ++hk) reduces.push_back({kv_off, nk, hk, part_base + hk * nparts, nparts, acc, {0, 0}});
      }
      for (int j = 0; j < nparts; ++j) {
        int64_t c0 = nparts > 1 ? j * chunk_rows : 0;
        int64_t c1 = nparts > 1 ? std::min(nq_total, (j + 1) * chunk_rows) : nq_total;
        BTask b;
        b.kv_off = kv_off;
        b.nk = nk;
        b.kv_pos0 = kv_pos0;
        b.q_off = (int32_t)(cons_off[m] + c0);
        b.nq = (int32_t)(c1 - c0);
        b.mask_lo = (int32_t)std::min<int64_t>(std::max<int64_t>(mlo - c0, 0), b.nq);
        b.mask_hi = (int32_t)std::min<int64_t>(std::max<int64_t>(mhi - c0, 0), b.nq);
        b.part_base = part_base;
        b.nparts = nparts;
        b.chunk = j;
        b.acc = acc;
        b.cost = (double)b.nq * nk + 4096.0;
        btasks.push_back(b);
      }
    }
    // sort key.  The tiles of a node with descendants that each take one chunk stream the same
    // consumer rows, the descendants' rows first.  They share the largest of their costs as key,
    // so that they stay one run through the longest-first sort, run at the same time and stream
    // those rows through L2 once (each tile sees 128 fewer of the node's own rows than the one
    // before it, so their own costs differ).  Every other task keeps its own cost: a leaf's tiles
    // share no rows beyond its own, and the chunks of a split tile are equal already.
    double node_key = 0.0;
    int64_t node_group = -1;
    auto grouped = [&](const BTask& b) { return b.nparts == 1 && desc_len[m] > 0; };
    for (size_t i = first_task; i < btasks.size(); ++i)
      if (grouped(btasks[i])) {
        node_key = std::max(node_key, btasks[i].cost);
        if (node_group < 0) node_group = (int64_t)i;
      }
    for (size_t i = first_task; i < btasks.size(); ++i) {
      const bool g = grouped(btasks[i]);
      btasks[i].key = g ? node_key : btasks[i].cost;
      btasks[i].group = g ? node_group : (int64_t)i;
    }
  }
  if (part_tiles > INT32_MAX / 2) return fail(PSATTN_E_UNSUPPORTED, "too many partial tiles");
  t->bkv_part_tiles = part_tiles;
  t->reduce = reduces;
  {
    // longest first by key; a group (equal keys can be several groups) stays one run, its tiles
    // in order
    std::vector<int> ord(btasks.size());
    std::iota(ord.begin(), ord.end(), 0);
    std::stable_sort(ord.begin(), ord.end(), [&](int x, int y) {
      if (btasks[x].key != btasks[y].key) return btasks[x].key > btasks[y].key;
      return btasks[x].group < btasks[y].group;
    });
    t->bkv.clear();
    for (int i : ord) {
      const BTask& b = btasks[i];
      for (int hk = 0; hk < t->hkv; ++hk) {
        int32_t part = b.nparts > 1 ? b.part_base + hk * b.nparts + b.chunk : -1;
        t->bkv.push_back({b.kv_off, b.nk, b.kv_pos0, b.q_off, b.nq, hk, part, b.mask_lo, b.mask_hi, b.acc});
      }
    }
  }

  // ---------------- slots of this call's blocks that hold no token ----------------
  // (the padding of internal nodes' blocks; the rest of the pool -- other trees, cached blocks --
  // is left untouched)
  t->pad_slots.clear();
  for (int n = 0; n < N; ++n) {
    if (t->ext[n]) continue;
    for (int b = t->blk_ptr[n]; b < t->blk_ptr[n + 1]; ++b)
      for (int k = t->blocks[b].len; k < t->blocks[b].capacity; ++k) t->pad_slots.push_back((int32_t)(t->blocks[b].base + k));
  }

  if (t->fwd.size() > (size_t)INT32_MAX || t->bkv.size() > (size_t)INT32_MAX)
    return fail(PSATTN_E_UNSUPPORTED, "too many work items");

  // sequence position of every q_list entry, so that kernels staging consumer rows need no
  // dependent load; the device copy is preceded by -1, the position of a row past a list
  t->q_pos.resize(t->q_list.size());
  for (size_t i = 0; i < t->q_list.size(); ++i) t->q_pos[i] = t->row_pos[t->q_list[i]];
  const int32_t past_list = -1;

  // ---------------- device image ----------------
  size_t cur = 0;
  auto place = [&](size_t bytes) {
    size_t at = cur;
    cur = align_up(cur + std::max<size_t>(bytes, 4));
    return at;
  };
  t->o_row_pos = place(t->row_pos.size() * 4);
  t->o_row_slot = place(t->row_slot.size() * 4);
  t->o_q = place(t->q_list.size() * 4);
  t->o_qpos = place((t->q_pos.size() + 1) * 4);
  t->o_kv = place(t->kv_list.size() * 4);
  t->o_fwd = place(t->fwd.size() * sizeof(FwdItem));
  t->o_merge = place(t->merge.size() * sizeof(MergeEntry));
  t->o_bkv = place(t->bkv.size() * sizeof(BkvItem));
  t->o_reduce = place(t->reduce.size() * sizeof(ReduceEntry));
  t->o_pad = place(t->pad_slots.size() * 4);
  t->plan_bytes = cur;
  t->image.assign(cur, 0);
  auto put = [&](size_t at, const void* p, size_t bytes) {
    if (bytes) memcpy(t->image.data() + at, p, bytes);
  };
  put(t->o_row_pos, t->row_pos.data(), t->row_pos.size() * 4);
  put(t->o_row_slot, t->row_slot.data(), t->row_slot.size() * 4);
  put(t->o_q, t->q_list.data(), t->q_list.size() * 4);
  put(t->o_qpos, &past_list, 4);
  put(t->o_qpos + 4, t->q_pos.data(), t->q_pos.size() * 4);
  put(t->o_kv, t->kv_list.data(), t->kv_list.size() * 4);
  put(t->o_fwd, t->fwd.data(), t->fwd.size() * sizeof(FwdItem));
  put(t->o_merge, t->merge.data(), t->merge.size() * sizeof(MergeEntry));
  put(t->o_bkv, t->bkv.data(), t->bkv.size() * sizeof(BkvItem));
  put(t->o_reduce, t->reduce.data(), t->reduce.size() * sizeof(ReduceEntry));
  put(t->o_pad, t->pad_slots.data(), t->pad_slots.size() * 4);
  return PSATTN_OK;
}

PlanView plan_view(const psattn_tree* t) {
  const uint8_t* b = (const uint8_t*)t->dev;
  PlanView v;
  v.row_pos = (const int32_t*)(b + t->o_row_pos);
  v.row_slot = (const int32_t*)(b + t->o_row_slot);
  v.q_list = (const int32_t*)(b + t->o_q);
  v.q_pos = (const int32_t*)(b + t->o_qpos) + 1;
  v.kv_list = (const int32_t*)(b + t->o_kv);
  v.fwd = (const FwdItem*)(b + t->o_fwd);
  v.merge = (const MergeEntry*)(b + t->o_merge);
  v.bkv = (const BkvItem*)(b + t->o_bkv);
  v.reduce = (const ReduceEntry*)(b + t->o_reduce);
  v.pad_slots = (const int32_t*)(b + t->o_pad);
  return v;
}

// workspace layouts
struct FwdWs { size_t o_part_o, o_part_lse, total; };
FwdWs fwd_ws(const psattn_tree* t) {
  FwdWs w;
  size_t cur = 0;
  w.o_part_o = cur;
  cur = align_up(cur + (size_t)t->fwd_part_rows * t->hq * t->d * 4);
  w.o_part_lse = cur;
  cur = align_up(cur + (size_t)t->fwd_part_rows * t->hq * 4);
  w.total = t->fwd_part_rows ? cur : 0;
  return w;
}
struct BwdWs { size_t o_delta, o_lse2, o_kv_nls, o_kv_nd, o_part_dq, o_part_eps, o_part_dk, o_part_dv, total; };
BwdWs bwd_ws(const psattn_tree* t) {
  BwdWs w;
  size_t cur = 0;
  w.o_delta = cur;
  cur = align_up(cur + (size_t)t->Ns * t->hq * 4);
  w.o_lse2 = cur;
  cur = align_up(cur + (size_t)t->Ns * t->hq * 4);
  w.o_kv_nls = cur;
  cur = align_up(cur + (size_t)t->Ns * t->hq * 4);
  w.o_kv_nd = cur;
  cur = align_up(cur + (size_t)t->Ns * t->hq * 4);
  w.o_part_dq = cur;
  cur = align_up(cur + (size_t)t->fwd_part_rows * t->hq * t->d * 4);
  w.o_part_eps = cur;
  cur = align_up(cur + (size_t)t->fwd_part_rows * t->hq * 4);
  w.o_part_dk = cur;
  cur = align_up(cur + (size_t)t->bkv_part_tiles * BKV_TILE * t->d * 4);
  w.o_part_dv = cur;
  cur = align_up(cur + (size_t)t->bkv_part_tiles * BKV_TILE * t->d * 4);
  w.total = cur;
  return w;
}

bool misaligned(const void* p) { return ((uintptr_t)p & 15) != 0; }

// ---------------------------------------------------------------------------------------------
// Kernel timing

struct ProfRec {
  int kernel;
  hipEvent_t a, b;
};
struct Profiler {
  bool on = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> spare;
};
Profiler g_prof;
const char* kKernelNames[] = {"fwd_main", "fwd_merge",     "bwd_pre", "bwd_kv",   "bwd_dq", "bwd_reduce_kv",
                              "bwd_reduce_dq", "bwd_zero_pad", "rope",    "kv_scatter", "kv_gather"};
constexpr int kNumKernels = 11;

hipEvent_t get_event() {
  if (!g_prof.spare.empty()) {
    hipEvent_t e = g_prof.spare.back();
    g_prof.spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
psattn_status timed(int kernel, hipStream_t st, F&& launch) {
  hipEvent_t a = nullptr, b = nullptr;
  if (g_prof.on) {
    a = get_event();
    b = get_event();
    if (a && b) (void)hipEventRecord(a, st);
  }
  hipError_t e = launch();
  if (e != hipSuccess) return fail(PSATTN_E_HIP, "%s launch failed: %s", kKernelNames[kernel], hipGetErrorString(e));
  if (g_prof.on && a && b) {
    (void)hipEventRecord(b, st);
    g_prof.recs.push_back({kernel, a, b});
  }
  return PSATTN_OK;
}

}  // namespace

// =============================================================================================
// C ABI

extern "C" {

psattn_status psattn_tree_create(const psattn_tree_desc* desc, const psattn_plan_opts* opts, psattn_tree** out) {
  if (!out) return fail(PSATTN_E_INVALID_ARG, "out is NULL");
  psattn_plan_opts o{};
  if (opts) {
    o = *opts;
    for (int i = 0; i < 5; ++i)
      if (o.reserved[i] != 0) return fail(PSATTN_E_INVALID_ARG, "psattn_plan_opts.reserved must be zero");
    if (o.num_cus < 0) return fail(PSATTN_E_INVALID_ARG, "num_cus must be >= 0");
  }
  psattn_tree* t = new (std::nothrow) psattn_tree();
  if (!t) return fail(PSATTN_E_INVALID_ARG, "out of host memory");
  psattn_status st;
  try {
    st = validate_and_copy(desc, t);
    if (st == PSATTN_OK) st = build_plan(t, o);
#ifdef PSATTN_PLAN_CHECKS
    if (st == PSATTN_OK) st = check_plan(t);
#endif
  } catch (const std::bad_alloc&) {
    st = fail(PSATTN_E_UNSUPPORTED, "out of host memory while planning");
  } catch (...) {
    st = fail(PSATTN_E_INVALID_ARG, "unexpected error while planning");
  }
  if (st != PSATTN_OK) {
    delete t;
    return st;
  }
  *out = t;
  return PSATTN_OK;
}

void psattn_tree_destroy(psattn_tree* tree) { delete tree; }

psattn_status psattn_tree_device_bytes(const psattn_tree* t, size_t* bytes) {
  if (!t || !bytes) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  *bytes = t->plan_bytes;
  return PSATTN_OK;
}

psattn_status psattn_tree_upload(psattn_tree* t, void* dev_buf, size_t bytes, void* stream) {
  if (!t || !dev_buf) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (((uintptr_t)dev_buf & (kAlign - 1)) != 0) return fail(PSATTN_E_ALIGNMENT, "plan buffer must be 256-byte aligned");
  if (bytes < t->plan_bytes)
    return fail(PSATTN_E_WORKSPACE, "plan buffer has %zu bytes, needs %zu", bytes, t->plan_bytes);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = hipMemcpyAsync(dev_buf, t->image.data(), t->plan_bytes, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(PSATTN_E_HIP, "plan upload failed: %s", hipGetErrorString(e));
  t->dev = dev_buf;
  t->dev_bytes = bytes;
  return PSATTN_OK;
}

psattn_status psattn_workspace_size(const psattn_tree* t, int pass, size_t* bytes) {
  if (!t || !bytes) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (pass == 0) *bytes = fwd_ws(t).total;
  else if (pass == 1) *bytes = bwd_ws(t).total;
  else return fail(PSATTN_E_INVALID_ARG, "pass must be 0 (fwd) or 1 (bwd)");
  return PSATTN_OK;
}

psattn_status psattn_fwd(const psattn_tree* t, const void* Q, const void* K, const void* V, void* O, float* LSE,
                         void* O_lo, void* ws, size_t ws_bytes, void* stream) {
  if (!t) return fail(PSATTN_E_INVALID_ARG, "tree is NULL");
  if (!t->dev) return fail(PSATTN_E_NOT_UPLOADED, "call psattn_tree_upload before psattn_fwd");
  if (!Q || !K || !V || !O || !LSE) return fail(PSATTN_E_INVALID_ARG, "NULL tensor pointer");
  if (O_lo && t->dtype != PSATTN_BF16) return fail(PSATTN_E_INVALID_ARG, "O_lo is for bf16 trees only (must be NULL)");
  if (misaligned(Q) || misaligned(K) || misaligned(V) || misaligned(O) || misaligned(LSE) || misaligned(O_lo))
    return fail(PSATTN_E_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  FwdWs w = fwd_ws(t);
  if (ws_bytes < w.total || (w.total && !ws))
    return fail(PSATTN_E_WORKSPACE, "forward workspace has %zu bytes, needs %zu", ws_bytes, w.total);
  if (w.total && misaligned(ws)) return fail(PSATTN_E_ALIGNMENT, "workspace must be 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  FwdArgs a;
  a.plan = plan_view(t);
  a.s = t->shape;
  a.n_items = (int32_t)t->fwd.size();
  a.n_merge = (int32_t)t->merge.size();
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.O = O;
  a.O_lo = O_lo;
  a.LSE = LSE;
  a.part_o = w.total ? (float*)((uint8_t*)ws + w.o_part_o) : nullptr;
  a.part_lse = w.total ? (float*)((uint8_t*)ws + w.o_part_lse) : nullptr;
  a.pool_slots = t->pool_slots;
  const bool bf16 = t->dtype == PSATTN_BF16;
  psattn_status s = timed(0, st, [&] { return launch_fwd_main(a, bf16, st); });
  if (s == PSATTN_OK && a.n_merge) s = timed(1, st, [&] { return launch_fwd_merge(a, bf16, st); });
  return s;
}

psattn_status psattn_bwd(const psattn_tree* t, const void* Q, const void* K, const void* V, const void* O,
                         const float* LSE, const void* O_lo, const void* dO, float* dQ, float* dK, float* dV, void* ws,
                         size_t ws_bytes, void* stream) {
  if (!t) return fail(PSATTN_E_INVALID_ARG, "tree is NULL");
  if (!t->dev) return fail(PSATTN_E_NOT_UPLOADED, "call psattn_tree_upload before psattn_bwd");
  if (!Q || !K || !V || !O || !LSE || !dO || !dQ || !dK || !dV) return fail(PSATTN_E_INVALID_ARG, "NULL tensor pointer");
  if (O_lo && t->dtype != PSATTN_BF16) return fail(PSATTN_E_INVALID_ARG, "O_lo is for bf16 trees only (must be NULL)");
  if (misaligned(Q) || misaligned(K) || misaligned(V) || misaligned(O) || misaligned(LSE) || misaligned(dO) ||
      misaligned(dQ) || misaligned(dK) || misaligned(dV) || misaligned(O_lo))
    return fail(PSATTN_E_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  BwdWs w = bwd_ws(t);
  if (!ws || ws_bytes < w.total)
    return fail(PSATTN_E_WORKSPACE, "backward workspace has %zu bytes, needs %zu", ws_bytes, w.total);
  if (misaligned(ws)) return fail(PSATTN_E_ALIGNMENT, "workspace must be 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  BwdArgs a;
  a.plan = plan_view(t);
  a.s = t->shape;
  a.n_fwd = (int32_t)t->fwd.size();
  a.n_merge = (int32_t)t->merge.size();
  a.n_bkv = (int32_t)t->bkv.size();
  a.n_reduce = (int32_t)t->reduce.size();
  a.n_pad = (int32_t)t->pad_slots.size();
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.O = O;
  a.O_lo = O_lo;
  a.LSE = LSE;
  a.dO = dO;
  a.dQ = dQ;
  a.dK = dK;
  a.dV = dV;
  uint8_t* wb = (uint8_t*)ws;
  a.delta = (float*)(wb + w.o_delta);
  a.lse2 = (float*)(wb + w.o_lse2);
  a.kv_nls = (float*)(wb + w.o_kv_nls);
  a.kv_nd = (float*)(wb + w.o_kv_nd);
  a.part_dq = (float*)(wb + w.o_part_dq);
  a.part_eps = (float*)(wb + w.o_part_eps);
  a.part_dk = (float*)(wb + w.o_part_dk);
  a.part_dv = (float*)(wb + w.o_part_dv);
  a.pool_slots = t->pool_slots;
  const bool bf16 = t->dtype == PSATTN_BF16;
  // dQ first: in bf16 mode it also turns Delta (from the bf16 O) into the exact sum_j P dP that the
  // dK/dV pass uses
  psattn_status s = timed(2, st, [&] { return launch_bwd_pre(a, bf16, st); });
  if (s == PSATTN_OK) s = timed(4, st, [&] { return launch_bwd_dq(a, bf16, st); });
  if (s == PSATTN_OK && a.n_merge) s = timed(6, st, [&] { return launch_bwd_reduce_dq(a, bf16, st); });
  if (s == PSATTN_OK) s = timed(3, st, [&] { return launch_bwd_kv(a, bf16, st); });
  if (s == PSATTN_OK && a.n_reduce) s = timed(5, st, [&] { return launch_bwd_reduce_kv(a, st); });
  if (s == PSATTN_OK && a.n_pad) s = timed(7, st, [&] { return launch_bwd_zero_pad(a, st); });
  return s;
}

// ---------------------------------------------------------------------------------------------
// Layer steps around the attention (the rest of a layer in the shared layout)

psattn_status psattn_rope(const psattn_tree* t, void* X, psattn_dtype dtype, int32_t heads, float theta, int32_t inverse,
                          void* stream) {
  if (!t || !X) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (dtype != PSATTN_BF16 && dtype != PSATTN_FP32) return fail(PSATTN_E_UNSUPPORTED, "unknown dtype %d", (int)dtype);
  if (!t->dev) return fail(PSATTN_E_NOT_UPLOADED, "call psattn_tree_upload before psattn_rope");
  if (heads < 1) return fail(PSATTN_E_INVALID_ARG, "heads must be >= 1 (got %d)", heads);
  if (!(theta > 1.f) || !std::isfinite(theta)) return fail(PSATTN_E_INVALID_ARG, "theta must be finite and > 1");
  if (misaligned(X)) return fail(PSATTN_E_ALIGNMENT, "X must be 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  return timed(8, st, [&] {
    return launch_rope(plan_view(t), (int32_t)t->Ns, heads, t->d, theta, inverse != 0, dtype == PSATTN_BF16, X, st);
  });
}

psattn_status psattn_kv_scatter(const psattn_tree* t, const void* K_rows, const void* V_rows, void* K, void* V,
                                void* stream) {
  if (!t || !K_rows || !V_rows || !K || !V) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (!t->dev) return fail(PSATTN_E_NOT_UPLOADED, "call psattn_tree_upload before psattn_kv_scatter");
  if (misaligned(K_rows) || misaligned(V_rows) || misaligned(K) || misaligned(V))
    return fail(PSATTN_E_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  const int32_t row_bytes = t->hkv * t->d * (t->dtype == PSATTN_BF16 ? 2 : 4);
  return timed(9, st, [&] { return launch_kv_move(plan_view(t), (int32_t)t->Ns, row_bytes, true, K_rows, V_rows, K, V, st); });
}

psattn_status psattn_kv_gather(const psattn_tree* t, const float* dK, const float* dV, float* dK_rows, float* dV_rows,
                               void* stream) {
  if (!t || !dK || !dV || !dK_rows || !dV_rows) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  if (!t->dev) return fail(PSATTN_E_NOT_UPLOADED, "call psattn_tree_upload before psattn_kv_gather");
  if (misaligned(dK) || misaligned(dV) || misaligned(dK_rows) || misaligned(dV_rows))
    return fail(PSATTN_E_ALIGNMENT, "tensor pointers must be 16-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  const int32_t row_bytes = t->hkv * t->d * 4;
  return timed(10, st, [&] {
    return launch_kv_move(plan_view(t), (int32_t)t->Ns, row_bytes, false, dK, dV, dK_rows, dV_rows, st);
  });
}

psattn_status psattn_tree_refcounts(const psattn_tree* t, int32_t* node_refcount) {
  if (!t || !node_refcount) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  std::copy(t->refcount.begin(), t->refcount.end(), node_refcount);
  return PSATTN_OK;
}

psattn_status psattn_tree_get_info(const psattn_tree* t, psattn_tree_info* info) {
  if (!t || !info) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  info->num_rows = t->Ns;
  info->unshared_tokens = t->Nu;
  info->visible_pairs = t->nvis;
  info->fwd_items = (int64_t)t->fwd.size();
  info->fwd_merges = (int64_t)t->merge.size();
  info->bkv_items = (int64_t)t->bkv.size();
  info->bkv_reduces = (int64_t)t->reduce.size();
  info->pad_slots = (int64_t)t->pad_slots.size();
  info->fwd_partial_rows = t->fwd_part_rows;
  info->bkv_partial_tiles = t->bkv_part_tiles;
  info->plan_bytes = (int64_t)t->plan_bytes;
  info->q_tile_rows = t->shape.bmq;
  info->kv_tile_keys = KV_TILE;
  info->bkv_tile_keys = BKV_TILE;
  info->head_chunk = t->shape.hc;
  return PSATTN_OK;
}

psattn_status psattn_tree_plan_array(const psattn_tree* t, int which, const int32_t** data, int64_t* count,
                                     int32_t* width) {
  if (!t || !data || !count || !width) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  switch (which) {
    case 0: *data = t->row_pos.data(); *count = (int64_t)t->row_pos.size(); *width = 1; break;
    case 1: *data = t->q_list.data(); *count = (int64_t)t->q_list.size(); *width = 1; break;
    case 2: *data = t->kv_list.data(); *count = (int64_t)t->kv_list.size(); *width = 1; break;
    case 3: *data = (const int32_t*)t->fwd.data(); *count = (int64_t)t->fwd.size(); *width = 8; break;
    case 4: *data = (const int32_t*)t->merge.data(); *count = (int64_t)t->merge.size(); *width = 4; break;
    case 5: *data = (const int32_t*)t->bkv.data(); *count = (int64_t)t->bkv.size(); *width = 10; break;
    case 6: *data = (const int32_t*)t->reduce.data(); *count = (int64_t)t->reduce.size(); *width = 8; break;
    case 7: *data = t->pad_slots.data(); *count = (int64_t)t->pad_slots.size(); *width = 1; break;
    case 8: *data = t->row_slot.data(); *count = (int64_t)t->row_slot.size(); *width = 1; break;
    case 9: *data = t->q_pos.data(); *count = (int64_t)t->q_pos.size(); *width = 1; break;
    default: return fail(PSATTN_E_INVALID_ARG, "unknown plan array %d", which);
  }
  return PSATTN_OK;
}

psattn_status psattn_profile_enable(int enable) {
  g_prof.on = enable != 0;
  return PSATTN_OK;
}

psattn_status psattn_profile_reset(void) {
  for (ProfRec& r : g_prof.recs) {
    g_prof.spare.push_back(r.a);
    g_prof.spare.push_back(r.b);
  }
  g_prof.recs.clear();
  return PSATTN_OK;
}

psattn_status psattn_profile_read(int32_t max_entries, int32_t* num_entries, const char** names, int64_t* launches,
                                  double* total_ms) {
  if (!num_entries) return fail(PSATTN_E_INVALID_ARG, "NULL argument");
  int64_t cnt[kNumKernels] = {0};
  double ms[kNumKernels] = {0};
  for (ProfRec& r : g_prof.recs) {
    hipError_t e = hipEventSynchronize(r.b);
    float x = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&x, r.a, r.b);
    if (e != hipSuccess) return fail(PSATTN_E_HIP, "reading kernel timers failed: %s", hipGetErrorString(e));
    cnt[r.kernel]++;
    ms[r.kernel] += x;
  }
  int n = 0;
  for (int k = 0; k < kNumKernels; ++k) {
    if (!cnt[k]) continue;
    if (n < max_entries) {
      if (names) names[n] = kKernelNames[k];
      if (launches) launches[n] = cnt[k];
      if (total_ms) total_ms[n] = ms[k];
    }
    ++n;
  }
  *num_entries = n;
  return PSATTN_OK;
}

const char* psattn_status_string(psattn_status s) {
  switch (s) {
    case PSATTN_OK: return "PSATTN_OK";
    case PSATTN_E_INVALID_ARG: return "PSATTN_E_INVALID_ARG";
    case PSATTN_E_INVALID_TREE: return "PSATTN_E_INVALID_TREE";
    case PSATTN_E_BLOCK_RANGE: return "PSATTN_E_BLOCK_RANGE";
    case PSATTN_E_BLOCK_OVERLAP: return "PSATTN_E_BLOCK_OVERLAP";
    case PSATTN_E_BLOCK_COVERAGE: return "PSATTN_E_BLOCK_COVERAGE";
    case PSATTN_E_UNSUPPORTED: return "PSATTN_E_UNSUPPORTED";
    case PSATTN_E_WORKSPACE: return "PSATTN_E_WORKSPACE";
    case PSATTN_E_ALIGNMENT: return "PSATTN_E_ALIGNMENT";
    case PSATTN_E_HIP: return "PSATTN_E_HIP";
    case PSATTN_E_NOT_UPLOADED: return "PSATTN_E_NOT_UPLOADED";
    case PSATTN_E_INTERNAL: return "PSATTN_E_INTERNAL";
  }
  return "PSATTN_E_UNKNOWN";
}

const char* psattn_last_error(void) { return g_err.c_str(); }

}  // extern "C"
