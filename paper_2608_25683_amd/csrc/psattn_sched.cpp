// Host scheduling of prefix-shared training work (Sec. 4.2 workload model and greedy placement,
// Sec. 4.3 token-wise micro-batching).
//
// Workload of one sequence s of length l whose first h tokens are already cached (Eq.
// "single_sequence"): T(s) = a1 * l_suf * l + a2 * l_suf + a3 with l_suf = l - h: attention of
// the l_suf new queries over up to l keys, the per-token layers, and a fixed overhead.  The
// coefficients come from profiling (psattn_sched_fit: least squares over measured runs).
// A semantic group's workload is the sum over its sequences, each counting as cached what the
// group's earlier sequences computed; groups are placed whole, longest first, on the least-loaded
// worker.  Within a worker, token-wise micro-batching cuts the sequences into micro-batches of
// about equal workload, splitting a sequence at a token boundary when it would overflow the
// current micro-batch; its remaining tokens continue in the next micro-batch with the part
// already done as cached prefix (self-sequence sharing).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <new>
#include <numeric>
#include <vector>

#include "psattn.h"

namespace psattn {
psattn_status set_error(psattn_status st, const char* msg);
}

namespace {

psattn_status sfail(psattn_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return psattn::set_error(st, buf);
}

double cost(const double a[3], double l_suf, double l) { return a[0] * l_suf * l + a[1] * l_suf + a[2]; }

psattn_status check_forest(int32_t N, const int32_t* parent, const int32_t* seg_len, int32_t S, const int32_t* end) {
  if (N < 1 || S < 1 || !parent || !seg_len || !end) return sfail(PSATTN_E_INVALID_ARG, "empty forest or NULL array");
  for (int i = 0; i < N; ++i) {
    if (parent[i] < -1 || parent[i] >= i)
      return sfail(PSATTN_E_INVALID_TREE, "parent[%d] = %d: a parent must precede its child (or be -1)", i, parent[i]);
    if (seg_len[i] < 1) return sfail(PSATTN_E_INVALID_TREE, "seg_len[%d] = %d: segments must be non-empty", i, seg_len[i]);
  }
  for (int s = 0; s < S; ++s)
    if (end[s] < 0 || end[s] >= N) return sfail(PSATTN_E_INVALID_TREE, "sample_end[%d] = %d out of range", s, end[s]);
  return PSATTN_OK;
}

std::vector<int32_t> path_of(const int32_t* parent, int e) {
  std::vector<int32_t> p;
  for (int n = e; n >= 0; n = parent[n]) p.push_back(n);
  std::reverse(p.begin(), p.end());
  return p;
}

}  // namespace

extern "C" psattn_status psattn_sched_fit(int32_t n, const double* l_suf, const double* l, const double* t,
                                          double alpha[3]) {
  if (n < 3 || !l_suf || !l || !t || !alpha) return sfail(PSATTN_E_INVALID_ARG, "need at least 3 measurements");
  // normal equations of min sum (x_i . a - t_i)^2 with x_i = (l_suf * l, l_suf, 1)
  double A[3][3] = {}, b[3] = {};
  for (int i = 0; i < n; ++i) {
    const double x[3] = {l_suf[i] * l[i], l_suf[i], 1.0};
    for (int r = 0; r < 3; ++r) {
      b[r] += x[r] * t[i];
      for (int c = 0; c < 3; ++c) A[r][c] += x[r] * x[c];
    }
  }
  // Gaussian elimination with partial pivoting
  int piv[3] = {0, 1, 2};
  for (int k = 0; k < 3; ++k) {
    int p = k;
    for (int r = k + 1; r < 3; ++r)
      if (std::fabs(A[r][k]) > std::fabs(A[p][k])) p = r;
    if (std::fabs(A[p][k]) < 1e-300) return sfail(PSATTN_E_INVALID_ARG, "measurements do not determine the 3 coefficients");
    std::swap(A[k], A[p]);
    std::swap(b[k], b[p]);
    std::swap(piv[k], piv[p]);
    for (int r = k + 1; r < 3; ++r) {
      const double f = A[r][k] / A[k][k];
      for (int c = k; c < 3; ++c) A[r][c] -= f * A[k][c];
      b[r] -= f * b[k];
    }
  }
  for (int k = 2; k >= 0; --k) {
    double s = b[k];
    for (int c = k + 1; c < 3; ++c) s -= A[k][c] * alpha[c];
    alpha[k] = s / A[k][k];
  }
  return PSATTN_OK;
}

extern "C" psattn_status psattn_sched_group_costs(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                                                  int32_t num_samples, const int32_t* sample_end,
                                                  const int32_t* group_of_sample, int32_t num_groups,
                                                  const double alpha[3], double* group_cost) {
  psattn_status st = check_forest(num_nodes, parent, seg_len, num_samples, sample_end);
  if (st != PSATTN_OK) return st;
  if (!group_of_sample || !alpha || !group_cost || num_groups < 1) return sfail(PSATTN_E_INVALID_ARG, "NULL argument");
  std::fill(group_cost, group_cost + num_groups, 0.0);
  std::vector<int32_t> done_by(num_nodes, -1);   // group whose earlier sample computed the node
  for (int s = 0; s < num_samples; ++s) {
    const int g = group_of_sample[s];
    if (g < 0 || g >= num_groups) return sfail(PSATTN_E_INVALID_ARG, "group_of_sample[%d] = %d out of range", s, g);
    double l = 0, h = 0;
    for (int n : path_of(parent, sample_end[s])) {
      l += seg_len[n];
      if (done_by[n] == g) h += seg_len[n];   // cached by the group's earlier sequences
      done_by[n] = g;
    }
    group_cost[g] += cost(alpha, l - h, l);
  }
  return PSATTN_OK;
}

extern "C" psattn_status psattn_sched_place(int32_t num_groups, const double* group_cost, int32_t num_workers,
                                            int32_t* worker_of_group, double* worker_load) {
  if (num_groups < 1 || num_workers < 1 || !group_cost || !worker_of_group)
    return sfail(PSATTN_E_INVALID_ARG, "need groups, workers and non-NULL arrays");
  std::vector<int> ord(num_groups);
  std::iota(ord.begin(), ord.end(), 0);
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) { return group_cost[a] > group_cost[b]; });
  std::vector<double> load(num_workers, 0.0);
  for (int g : ord) {
    const int w = (int)(std::min_element(load.begin(), load.end()) - load.begin());   // lowest index on ties
    worker_of_group[g] = w;
    load[w] += group_cost[g];
  }
  if (worker_load) std::copy(load.begin(), load.end(), worker_load);
  return PSATTN_OK;
}

// ---------------------------------------------------------------------------------------------
// Token-wise micro-batching

struct psattn_sched_mb {
  std::vector<int32_t> parent, seg_len, src_node, src_off;   // refined forest
  std::vector<int32_t> chunk_end, chunk_mb, chunk_sample;    // one sample per chunk
  std::vector<double> mb_cost;
};

namespace {

psattn_status microbatch(psattn_sched_mb* m, int32_t N, const int32_t* parent, const int32_t* seg_len, int32_t S,
                         const int32_t* end, const double a[3], int32_t M) {
  // total workload of the worker's sequences in order (a sequence's cached prefix: what the
  // earlier sequences computed), and the per-micro-batch budget
  std::vector<char> done(N, 0);
  double total = 0;
  for (int s = 0; s < S; ++s) {
    double l = 0, h = 0;
    for (int n : path_of(parent, end[s])) {
      l += seg_len[n];
      if (done[n]) h += seg_len[n];
      done[n] = 1;
    }
    total += cost(a, l - h, l);
  }
  const double budget = total / M;
  // walk the sequences; cut positions per node (token offsets where a chunk ends inside a node)
  std::fill(done.begin(), done.end(), 0);
  std::vector<std::vector<int32_t>> cuts(N);
  struct Chunk { int node, off, mb, sample; };   // chunk ends after token off-1 of node
  std::vector<Chunk> chunks;
  int mb = 0;
  double used = 0;
  std::vector<double> mb_cost(M, 0.0);
  std::vector<int32_t> comp(N, 0);   // tokens of each node computed so far
  for (int s = 0; s < S; ++s) {
    const std::vector<int32_t> path = path_of(parent, end[s]);
    // positions along the path: tokens before node k, and the first token not yet computed
    int64_t l = 0, h = 0;
    for (int n : path) l += seg_len[n];
    {
      int64_t pos = 0;
      for (int n : path) {
        if (comp[n] == seg_len[n]) {
          pos += seg_len[n];
          continue;
        }
        pos += comp[n];
        break;
      }
      h = pos;
    }
    while (h < l) {
      // tokens x of the suffix that fit what is left of this micro-batch's budget (the last
      // micro-batch takes everything that remains)
      const double left = budget - used;
      int64_t x = l - h;
      if (mb < M - 1 && cost(a, (double)x, (double)l) > left) {
        // largest x with a1 x (h + x) + a2 x + a3 <= left
        const double qa = a[0], qb = a[0] * (double)h + a[1], qc = a[2] - left;
        double r;
        if (qa > 0) r = (-qb + std::sqrt(std::max(0.0, qb * qb - 4 * qa * qc))) / (2 * qa);
        else r = qb > 0 ? -qc / qb : 0.0;
        x = std::max<int64_t>(0, std::min<int64_t>(l - h, (int64_t)std::floor(r)));
        while (x > 0 && cost(a, (double)x, (double)(h + x)) > left) --x;
        if (x == 0) {   // nothing fits: close this micro-batch
          ++mb;
          used = 0;
          continue;
        }
      }
      // place tokens [h, h + x) of the path into micro-batch mb
      int64_t pos = 0, want = h + x;
      int cut_node = -1, cut_off = 0;
      for (int n : path) {
        const int64_t n0 = pos, n1 = pos + seg_len[n];
        if (want > n0 && h < n1) {
          const int32_t upto = (int32_t)(std::min(want, n1) - n0);
          comp[n] = std::max(comp[n], upto);
          if (want <= n1) {
            cut_node = n;
            cut_off = upto;
          }
        }
        pos = n1;
      }
      const double c = cost(a, (double)x, (double)(h + x));
      used += c;
      mb_cost[mb] += c;
      if (cut_off < seg_len[cut_node]) cuts[cut_node].push_back(cut_off);
      chunks.push_back({cut_node, cut_off, mb, s});
      h += x;
      if (h < l && mb < M - 1) {   // the sequence continues in the next micro-batch
        ++mb;
        used = 0;
      }
    }
  }
  // refined forest: node n becomes pieces [0, c1), [c1, c2), ..., each the parent of the next;
  // n's children hang below its last piece
  std::vector<int32_t> first(N), last(N);
  for (int n = 0; n < N; ++n) {
    std::vector<int32_t>& c = cuts[n];
    std::sort(c.begin(), c.end());
    c.erase(std::unique(c.begin(), c.end()), c.end());
    int32_t prev = 0;
    first[n] = (int32_t)m->parent.size();
    std::vector<int32_t> ends = c;
    ends.push_back(seg_len[n]);
    for (int32_t e : ends) {
      const int32_t par = prev == 0 ? (parent[n] < 0 ? -1 : last[parent[n]]) : (int32_t)m->parent.size() - 1;
      m->parent.push_back(par);
      m->seg_len.push_back(e - prev);
      m->src_node.push_back(n);
      m->src_off.push_back(prev);
      prev = e;
    }
    last[n] = (int32_t)m->parent.size() - 1;
  }
  // micro-batches that received a chunk, numbered in order (one that nothing fitted is dropped)
  std::vector<int32_t> renum(M, -1);
  for (const Chunk& ch : chunks) renum[ch.mb] = 0;
  int32_t k = 0;
  for (int i = 0; i < M; ++i)
    if (renum[i] == 0) {
      renum[i] = k++;
      m->mb_cost.push_back(mb_cost[i]);
    }
  for (const Chunk& ch : chunks) {
    // the refined piece of node ch.node that ends at token ch.off
    int32_t r = first[ch.node];
    while (m->src_off[r] + m->seg_len[r] != ch.off) ++r;
    m->chunk_end.push_back(r);
    m->chunk_mb.push_back(renum[ch.mb]);
    m->chunk_sample.push_back(ch.sample);
  }
  return PSATTN_OK;
}

}  // namespace

extern "C" psattn_status psattn_sched_microbatch(int32_t num_nodes, const int32_t* parent, const int32_t* seg_len,
                                                 int32_t num_samples, const int32_t* sample_end,
                                                 const double alpha[3], int32_t num_micro_batches,
                                                 psattn_sched_mb** out) {
  if (!out) return sfail(PSATTN_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  psattn_status st = check_forest(num_nodes, parent, seg_len, num_samples, sample_end);
  if (st != PSATTN_OK) return st;
  if (!alpha || num_micro_batches < 1) return sfail(PSATTN_E_INVALID_ARG, "need alpha and num_micro_batches >= 1");
  if (alpha[0] < 0 || alpha[1] < 0 || alpha[2] < 0 || alpha[0] + alpha[1] <= 0)
    return sfail(PSATTN_E_INVALID_ARG, "coefficients must be non-negative with a1 + a2 > 0");
  psattn_sched_mb* m = new (std::nothrow) psattn_sched_mb;
  if (!m) return sfail(PSATTN_E_INVALID_ARG, "out of host memory");
  try {
    st = microbatch(m, num_nodes, parent, seg_len, num_samples, sample_end, alpha, num_micro_batches);
  } catch (const std::bad_alloc&) {
    st = sfail(PSATTN_E_INVALID_ARG, "out of host memory");
  }
  if (st != PSATTN_OK) {
    delete m;
    return st;
  }
  *out = m;
  return PSATTN_OK;
}

extern "C" void psattn_sched_mb_destroy(psattn_sched_mb* m) { delete m; }

extern "C" psattn_status psattn_sched_mb_get(const psattn_sched_mb* m, psattn_sched_mb_view* v) {
  if (!m || !v) return sfail(PSATTN_E_INVALID_ARG, "NULL argument");
  v->num_nodes = (int32_t)m->parent.size();
  v->parent = m->parent.data();
  v->seg_len = m->seg_len.data();
  v->src_node = m->src_node.data();
  v->src_offset = m->src_off.data();
  v->num_chunks = (int32_t)m->chunk_end.size();
  v->chunk_end = m->chunk_end.data();
  v->chunk_micro_batch = m->chunk_mb.data();
  v->chunk_sample = m->chunk_sample.data();
  v->num_micro_batches = (int32_t)m->mb_cost.size();
  v->micro_batch_cost = m->mb_cost.data();
  return PSATTN_OK;
}
