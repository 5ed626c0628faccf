// HIP kernels for prefix-shared causal attention on CDNA4 (gfx950).
//
// bf16 path: v_mfma_f32_32x32x16_bf16 for every contraction.  The forward
// and dQ kernels compute the transposed score tile S^T = K Q^T so that each
// lane owns one query row (its column of S^T): softmax statistics are
// per-lane scalars, the only cross-lane step is one swap between the two
// 32-lane halves, and the probability tile feeds the next MFMA straight
// from the accumulator registers.  Key tiles are gathered through the plan's
// slot lists (one 256-byte row per key and head, fully coalesced) and staged
// in LDS; operands that must run along keys (V^T, K^T) or along query rows
// (Q^T, dO^T) are transposed while staging.  The dK/dV kernel keeps its keys
// stationary in registers and streams every consuming query row (the key's
// own later rows and all rows of all descendant branches) through LDS.
//
// fp32 path: plain VALU kernels with the same work items (true fp32 products
// and accumulation; no reduced-precision matrix formats).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "psattn_launch.h"

namespace psattn {
namespace {

typedef uint16_t bf16_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 as_bf(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }
__device__ __forceinline__ u32x2 ld8(const void* p) { return *(const u32x2*)p; }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}
__device__ __forceinline__ float bf2f(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
// 8 consecutive accumulator values -> one bf16x8 MFMA operand
__device__ __forceinline__ bf16x8 pack8(const f32x16& x, int base) {
  u32x4 w;
  w[0] = pack2(x[base + 0], x[base + 1]);
  w[1] = pack2(x[base + 2], x[base + 3]);
  w[2] = pack2(x[base + 4], x[base + 5]);
  w[3] = pack2(x[base + 6], x[base + 7]);
  return as_bf(w);
}
// interleave two rows' 8-element chunks into 8 dwords (row a in the low halves)
__device__ __forceinline__ void interleave(const u32x4& ra, const u32x4& rb, uint32_t* w) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    w[2 * e] = (ra[e] & 0xffffu) | (rb[e] << 16);
    w[2 * e + 1] = (ra[e] >> 16) | (rb[e] & 0xffff0000u);
  }
}

// ============================================================================================
// Forward, bf16.  One workgroup = one FwdItem: up to 32*rw query rows x hc heads x a key range.
// Wave w handles head head0 + w / rw, rows 32*(w % rw) .. +31.

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int T = NW * 64;
  constexpr int KS = D / 16;                                  // MFMA k-steps over head_dim
  constexpr int DB = D / 32;                                  // 32-wide blocks of head_dim
  constexpr int KSTR = D + 8;                                 // LDS row stride of K (elements)
  constexpr int VSTR = KV_TILE + 4;                           // LDS row stride of V^T (elements)
  constexpr int CPR = D / 8;                                  // 16-byte chunks per row
  constexpr int KCH = (KV_TILE * CPR + T - 1) / T;            // K chunks staged per thread
  constexpr int VUN = ((KV_TILE / 2) * CPR + T - 1) / T;      // V row-pair units per thread
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KV_TILE * KSTR];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VSTR];

  const FwdItem it = a.plan.fwd[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int rw = a.s.rw;
  const int head = it.head0 + wave / rw;
  const int hk = it.head0 / a.s.g;
  const int ridx = (wave % rw) * 32 + l32;
  const bool row_ok = ridx < it.nq;
  const int row = a.plan.q_list[it.q_off + (row_ok ? ridx : it.nq - 1)];
  const int qpos = a.plan.row_pos[row];

  bf16x8 qreg[KS];
  {
    const bf16_t* qp = (const bf16_t*)a.Q + ((size_t)row * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) qreg[s] = as_bf(ld16(qp + 16 * s));
  }

  const size_t kv_stride = (size_t)a.s.hkv * D;
  const bf16_t* Kb = (const bf16_t*)a.K + (size_t)hk * D;
  const bf16_t* Vb = (const bf16_t*)a.V + (size_t)hk * D;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int nkv = it.nkv;
  const int ntiles = (nkv + KV_TILE - 1) / KV_TILE;

  u32x4 kpre[KCH];
  u32x4 vpre[VUN][2];
  auto load_tile = [&](int t) {
    const int base = t * KV_TILE;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * T;
      if (c < KV_TILE * CPR) {
        const int key = min(base + c / CPR, nkv - 1);
        kpre[i] = ld16(Kb + (size_t)kvl[key] * kv_stride + (c % CPR) * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < VUN; ++i) {
      const int u = tid + i * T;
      if (u < (KV_TILE / 2) * CPR) {
        const int p = u / CPR, cc = u % CPR;
        const int k0 = min(base + 2 * p, nkv - 1), k1 = min(base + 2 * p + 1, nkv - 1);
        vpre[i][0] = ld16(Vb + (size_t)kvl[k0] * kv_stride + cc * 8);
        vpre[i][1] = ld16(Vb + (size_t)kvl[k1] * kv_stride + cc * 8);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * T;
      if (c < KV_TILE * CPR) *(u32x4*)&Ks[(c / CPR) * KSTR + (c % CPR) * 8] = kpre[i];
    }
#pragma unroll
    for (int i = 0; i < VUN; ++i) {
      const int u = tid + i * T;
      if (u < (KV_TILE / 2) * CPR) {
        const int p = u / CPR, cc = u % CPR;
        uint32_t w[8];
        interleave(vpre[i][0], vpre[i][1], w);
#pragma unroll
        for (int e = 0; e < 8; ++e) *(uint32_t*)&Vt[(cc * 8 + e) * VSTR + 2 * p] = w[e];
      }
    }
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int mb = 0; mb < DB; ++mb) oacc[mb] = f32x16{};
  float m_run = kNegInf, l_run = 0.f;
  const float c = a.s.scale * kLog2e;

  load_tile(0);
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (t + 1 < ntiles) load_tile(t + 1);

    f32x16 sacc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      sacc[b] = f32x16{};
#pragma unroll
      for (int s = 0; s < KS; ++s)
        sacc[b] = mfma(as_bf(ld16(&Ks[(32 * b + l32) * KSTR + 16 * s + 8 * hh])), qreg[s], sacc[b]);
    }
    if (t >= it.nfull) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kidx = t * KV_TILE + 32 * b + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (kidx >= nkv || it.kv_pos0 + kidx > qpos) sacc[b][v] = kNegInf;
        }
    }
    float mloc = kNegInf;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) mloc = fmaxf(mloc, sacc[b][v]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = fast_exp2((m_run - m_use) * c);
    const float mc = m_use * c;
    float psum = 0.f;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = fast_exp2(fmaf(sacc[b][v], c, -mc));
        sacc[b][v] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v) oacc[mb][v] *= alpha;

    bf16x8 pb[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      pb[b][0] = pack8(sacc[b], 0);
      pb[b][1] = pack8(sacc[b], 8);
    }
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const bf16_t* vp = &Vt[(32 * mb + l32) * VSTR + 32 * b + 16 * t2 + 4 * hh];
          const u32x2 lo = ld8(vp), hi = ld8(vp + 8);
          oacc[mb] = mfma(as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), pb[b][t2], oacc[mb]);
        }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse = l_tot > 0.f ? m_run * a.s.scale + logf(l_tot) : kNegInf;
  if (!row_ok) return;
  if (it.part < 0) {
    bf16_t* op = (bf16_t*)a.O + ((size_t)row * a.s.hq + head) * D;
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        u32x2 w;
        w[0] = pack2(oacc[mb][4 * g4 + 0] * inv, oacc[mb][4 * g4 + 1] * inv);
        w[1] = pack2(oacc[mb][4 * g4 + 2] * inv, oacc[mb][4 * g4 + 3] * inv);
        *(u32x2*)(op + 32 * mb + 8 * g4 + 4 * hh) = w;
      }
    if (hh == 0) a.LSE[(size_t)head * a.s.ns + row] = lse;
  } else {
    const size_t prow = (size_t)it.part + ridx;
    float* op = a.part_o + (prow * a.s.hq + head) * D;
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(f32x4*)(op + 32 * mb + 8 * g4 + 4 * hh) =
            f32x4{oacc[mb][4 * g4] * inv, oacc[mb][4 * g4 + 1] * inv, oacc[mb][4 * g4 + 2] * inv, oacc[mb][4 * g4 + 3] * inv};
    if (hh == 0) a.part_lse[prow * a.s.hq + head] = lse;
  }
}

// ============================================================================================
// Backward dK/dV, bf16.  One workgroup = one BkvItem: up to 128 keys of one kv head (wave w owns
// keys 32w..32w+31) x a chunk of consuming query rows, for every query head of the group.

template <int D>
__global__ __launch_bounds__(256) void bwd_kv_bf16_kernel(BwdArgs a) {
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int RSTR = D + 8;        // row-major query tile stride (elements)
  constexpr int TSTR = Q_SUB + 4;    // transposed query tile stride (elements)
  constexpr int CPR = D / 8;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[Q_SUB * RSTR];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[Q_SUB * RSTR];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[D * TSTR];
  __shared__ __attribute__((aligned(16))) bf16_t dOt[D * TSTR];
  __shared__ float s_lse[Q_SUB], s_del[Q_SUB];
  __shared__ int s_qpos[Q_SUB];
  __shared__ int s_slot[BKV_TILE];

  const BkvItem it = a.plan.bkv[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int hk = it.hk;
  const int G = a.s.g;
  const size_t kv_stride = (size_t)a.s.hkv * D;
  if (tid < BKV_TILE) s_slot[tid] = a.plan.kv_list[it.kv_off + min(tid, it.nk - 1)];

  const int kidx = 32 * wave + l32;
  const int kpos = it.kv_pos0 + kidx;
  bf16x8 kreg[KS], vreg[KS];
  {
    const int slot = a.plan.kv_list[it.kv_off + min(kidx, it.nk - 1)];
    const bf16_t* kp = (const bf16_t*)a.K + (size_t)slot * kv_stride + (size_t)hk * D + 8 * hh;
    const bf16_t* vp = (const bf16_t*)a.V + (size_t)slot * kv_stride + (size_t)hk * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kreg[s] = as_bf(ld16(kp + 16 * s));
      vreg[s] = as_bf(ld16(vp + 16 * s));
    }
  }
  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int nb = 0; nb < DB; ++nb) {
    dk[nb] = f32x16{};
    dv[nb] = f32x16{};
  }

  const int* ql = a.plan.q_list + it.q_off;
  const int nq = it.nq;
  const int nsub = (nq + Q_SUB - 1) / Q_SUB;
  const int nsteps = nsub * G;
  const bool stager = tid < (Q_SUB / 2) * CPR;
  const int sp = tid / CPR, scc = tid % CPR;   // staged row pair and 16-byte column chunk
  u32x4 qa, qb, da, db;
  float pre_lse = 0.f, pre_del = 0.f;
  int pre_qpos = -1;
  auto load_step = [&](int step) {
    const int sub = step / G, head = hk * G + step % G;
    if (stager) {
      const int r0 = min(Q_SUB * sub + 2 * sp, nq - 1), r1 = min(Q_SUB * sub + 2 * sp + 1, nq - 1);
      const size_t o0 = ((size_t)ql[r0] * a.s.hq + head) * D + scc * 8;
      const size_t o1 = ((size_t)ql[r1] * a.s.hq + head) * D + scc * 8;
      qa = ld16((const bf16_t*)a.Q + o0);
      qb = ld16((const bf16_t*)a.Q + o1);
      da = ld16((const bf16_t*)a.dO + o0);
      db = ld16((const bf16_t*)a.dO + o1);
    }
    if (tid < Q_SUB) {
      const int r = Q_SUB * sub + tid;
      const int row = ql[min(r, nq - 1)];
      pre_lse = a.LSE[(size_t)head * a.s.ns + row];
      pre_del = a.delta[(size_t)head * a.s.ns + row];
      pre_qpos = r < nq ? a.plan.row_pos[row] : -1;
    }
  };
  auto store_step = [&]() {
    if (stager) {
      *(u32x4*)&Qs[(2 * sp) * RSTR + scc * 8] = qa;
      *(u32x4*)&Qs[(2 * sp + 1) * RSTR + scc * 8] = qb;
      *(u32x4*)&dOs[(2 * sp) * RSTR + scc * 8] = da;
      *(u32x4*)&dOs[(2 * sp + 1) * RSTR + scc * 8] = db;
      uint32_t w[8];
      interleave(qa, qb, w);
#pragma unroll
      for (int e = 0; e < 8; ++e) *(uint32_t*)&Qt[(scc * 8 + e) * TSTR + 2 * sp] = w[e];
      interleave(da, db, w);
#pragma unroll
      for (int e = 0; e < 8; ++e) *(uint32_t*)&dOt[(scc * 8 + e) * TSTR + 2 * sp] = w[e];
    }
    if (tid < Q_SUB) {
      s_lse[tid] = pre_lse * kLog2e;
      s_del[tid] = pre_del;
      s_qpos[tid] = pre_qpos;
    }
  };

  const float c = a.s.scale * kLog2e;
  load_step(0);
  for (int step = 0; step < nsteps; ++step) {
    const int sub = step / G;
    __syncthreads();
    store_step();
    __syncthreads();
    if (step + 1 < nsteps) load_step(step + 1);

    // S = Q K^T and dP = dO V^T for 32 rows x this wave's 32 keys
    f32x16 S = f32x16{}, dP = f32x16{};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      S = mfma(as_bf(ld16(&Qs[l32 * RSTR + 16 * s + 8 * hh])), kreg[s], S);
      dP = mfma(as_bf(ld16(&dOs[l32 * RSTR + 16 * s + 8 * hh])), vreg[s], dP);
    }
    const bool need_mask = (Q_SUB * sub < it.nmask) || (Q_SUB * sub + Q_SUB > nq);
    // accumulator layout: lane <-> key (column), element v <-> row 8*(v/4) + 4*hh + v%4
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int qr = 8 * (v >> 2) + 4 * hh + (v & 3);
      float p = fast_exp2(fmaf(S[v], c, -s_lse[qr]));
      if (need_mask && kpos > s_qpos[qr]) p = 0.f;
      S[v] = p;
      dP[v] = p * (dP[v] - s_del[qr]);
    }
    const bf16x8 pa0 = pack8(S, 0), pa1 = pack8(S, 8);
    const bf16x8 sa0 = pack8(dP, 0), sa1 = pack8(dP, 8);
#pragma unroll
    for (int nb = 0; nb < DB; ++nb) {
      const int drow = (32 * nb + l32) * TSTR + 4 * hh;
      u32x2 lo = ld8(&dOt[drow]), hi = ld8(&dOt[drow + 8]);
      dv[nb] = mfma(pa0, as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), dv[nb]);
      lo = ld8(&dOt[drow + 16]);
      hi = ld8(&dOt[drow + 24]);
      dv[nb] = mfma(pa1, as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), dv[nb]);
      lo = ld8(&Qt[drow]);
      hi = ld8(&Qt[drow + 8]);
      dk[nb] = mfma(sa0, as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), dk[nb]);
      lo = ld8(&Qt[drow + 16]);
      hi = ld8(&Qt[drow + 24]);
      dk[nb] = mfma(sa1, as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), dk[nb]);
    }
  }

  // accumulator layout: lane <-> head_dim column 32*nb + l32, element v <-> key row of the wave
  const float scale = a.s.scale;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int key = 32 * wave + 8 * (v >> 2) + 4 * hh + (v & 3);
    if (key >= it.nk) continue;
    float* kdst;
    float* vdst;
    if (it.part < 0) {
      const size_t o = (size_t)s_slot[key] * kv_stride + (size_t)hk * D;
      kdst = a.dK + o;
      vdst = a.dV + o;
    } else {
      const size_t o = ((size_t)it.part * BKV_TILE + key) * D;
      kdst = a.part_dk + o;
      vdst = a.part_dv + o;
    }
#pragma unroll
    for (int nb = 0; nb < DB; ++nb) {
      kdst[32 * nb + l32] = dk[nb][v] * scale;
      vdst[32 * nb + l32] = dv[nb][v];
    }
  }
}

// ============================================================================================
// Backward dQ, bf16.  Same items and wave layout as the forward kernel.

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_dq_bf16_kernel(BwdArgs a) {
  constexpr int T = NW * 64;
  constexpr int KS = D / 16;
  constexpr int DB = D / 32;
  constexpr int KSTR = D + 8;
  constexpr int TSTR = KV_TILE + 4;
  constexpr int CPR = D / 8;
  constexpr int KUN = ((KV_TILE / 2) * CPR + T - 1) / T;   // K row-pair units per thread
  constexpr int VCH = (KV_TILE * CPR + T - 1) / T;         // V chunks per thread
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KV_TILE * KSTR];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[KV_TILE * KSTR];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[D * TSTR];

  const FwdItem it = a.plan.fwd[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int rw = a.s.rw;
  const int head = it.head0 + wave / rw;
  const int hk = it.head0 / a.s.g;
  const int ridx = (wave % rw) * 32 + l32;
  const bool row_ok = ridx < it.nq;
  const int row = a.plan.q_list[it.q_off + (row_ok ? ridx : it.nq - 1)];
  const int qpos = a.plan.row_pos[row];
  const float lse2 = a.LSE[(size_t)head * a.s.ns + row] * kLog2e;
  const float del = a.delta[(size_t)head * a.s.ns + row];

  bf16x8 qreg[KS], doreg[KS];
  {
    const size_t o = ((size_t)row * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qreg[s] = as_bf(ld16((const bf16_t*)a.Q + o + 16 * s));
      doreg[s] = as_bf(ld16((const bf16_t*)a.dO + o + 16 * s));
    }
  }
  const size_t kv_stride = (size_t)a.s.hkv * D;
  const bf16_t* Kb = (const bf16_t*)a.K + (size_t)hk * D;
  const bf16_t* Vb = (const bf16_t*)a.V + (size_t)hk * D;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int nkv = it.nkv;
  const int ntiles = (nkv + KV_TILE - 1) / KV_TILE;

  u32x4 kpre[KUN][2];
  u32x4 vpre[VCH];
  auto load_tile = [&](int t) {
    const int base = t * KV_TILE;
#pragma unroll
    for (int i = 0; i < KUN; ++i) {
      const int u = tid + i * T;
      if (u < (KV_TILE / 2) * CPR) {
        const int p = u / CPR, cc = u % CPR;
        const int k0 = min(base + 2 * p, nkv - 1), k1 = min(base + 2 * p + 1, nkv - 1);
        kpre[i][0] = ld16(Kb + (size_t)kvl[k0] * kv_stride + cc * 8);
        kpre[i][1] = ld16(Kb + (size_t)kvl[k1] * kv_stride + cc * 8);
      }
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int cidx = tid + i * T;
      if (cidx < KV_TILE * CPR) {
        const int key = min(base + cidx / CPR, nkv - 1);
        vpre[i] = ld16(Vb + (size_t)kvl[key] * kv_stride + (cidx % CPR) * 8);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KUN; ++i) {
      const int u = tid + i * T;
      if (u < (KV_TILE / 2) * CPR) {
        const int p = u / CPR, cc = u % CPR;
        *(u32x4*)&Ks[(2 * p) * KSTR + cc * 8] = kpre[i][0];
        *(u32x4*)&Ks[(2 * p + 1) * KSTR + cc * 8] = kpre[i][1];
        uint32_t w[8];
        interleave(kpre[i][0], kpre[i][1], w);
#pragma unroll
        for (int e = 0; e < 8; ++e) *(uint32_t*)&Kt[(cc * 8 + e) * TSTR + 2 * p] = w[e];
      }
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      const int cidx = tid + i * T;
      if (cidx < KV_TILE * CPR) *(u32x4*)&Vs[(cidx / CPR) * KSTR + (cidx % CPR) * 8] = vpre[i];
    }
  };

  f32x16 dq[DB];
#pragma unroll
  for (int mb = 0; mb < DB; ++mb) dq[mb] = f32x16{};
  const float c = a.s.scale * kLog2e;

  load_tile(0);
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (t + 1 < ntiles) load_tile(t + 1);

    f32x16 S[2], dP[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      S[b] = f32x16{};
      dP[b] = f32x16{};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        S[b] = mfma(as_bf(ld16(&Ks[(32 * b + l32) * KSTR + 16 * s + 8 * hh])), qreg[s], S[b]);
        dP[b] = mfma(as_bf(ld16(&Vs[(32 * b + l32) * KSTR + 16 * s + 8 * hh])), doreg[s], dP[b]);
      }
    }
    const bool need_mask = t >= it.nfull;
    // accumulator layout: lane <-> query row (column), element v <-> key 32*b + 8*(v/4) + 4*hh + v%4
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float p = fast_exp2(fmaf(S[b][v], c, -lse2));
        if (need_mask) {
          const int kidx = t * KV_TILE + 32 * b + 8 * (v >> 2) + 4 * hh + (v & 3);
          if (kidx >= nkv || it.kv_pos0 + kidx > qpos) p = 0.f;
        }
        dP[b][v] = p * (dP[b][v] - del);
      }
    bf16x8 sb[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      sb[b][0] = pack8(dP[b], 0);
      sb[b][1] = pack8(dP[b], 8);
    }
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2) {
          const bf16_t* kp = &Kt[(32 * mb + l32) * TSTR + 32 * b + 16 * t2 + 4 * hh];
          const u32x2 lo = ld8(kp), hi = ld8(kp + 8);
          dq[mb] = mfma(as_bf(u32x4{lo[0], lo[1], hi[0], hi[1]}), sb[b][t2], dq[mb]);
        }
  }

  if (!row_ok) return;
  const float scale = a.s.scale;
  float* dst = it.part < 0 ? a.dQ + ((size_t)row * a.s.hq + head) * D
                           : a.part_dq + (((size_t)it.part + ridx) * a.s.hq + head) * D;
#pragma unroll
  for (int mb = 0; mb < DB; ++mb)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *(f32x4*)(dst + 32 * mb + 8 * g4 + 4 * hh) = f32x4{dq[mb][4 * g4] * scale, dq[mb][4 * g4 + 1] * scale,
                                                          dq[mb][4 * g4 + 2] * scale, dq[mb][4 * g4 + 3] * scale};
}

// ============================================================================================
// fp32 path (VALU).  Two lanes per (row, head) pair, each holding half of head_dim.

template <int D>
__global__ __launch_bounds__(512) void fwd_f32_kernel(FwdArgs a) {
  constexpr int H = D / 2;
  constexpr int KP = D + 1;   // LDS row stride (floats)
  __shared__ float Kf[KV_TILE * KP];
  __shared__ float Vf[KV_TILE * KP];
  const FwdItem it = a.plan.fwd[blockIdx.x];
  const int tid = threadIdx.x, T = blockDim.x;
  const int pair = tid >> 1, half = tid & 1;
  const int head = it.head0 + pair / a.s.bmq;
  const int hk = it.head0 / a.s.g;
  const int ridx = pair % a.s.bmq;
  const bool row_ok = ridx < it.nq;
  const int row = a.plan.q_list[it.q_off + (row_ok ? ridx : it.nq - 1)];
  const int qpos = a.plan.row_pos[row];
  float q[H], o[H];
  const float* qp = (const float*)a.Q + ((size_t)row * a.s.hq + head) * D + half * H;
#pragma unroll
  for (int i = 0; i < H; ++i) {
    q[i] = qp[i];
    o[i] = 0.f;
  }
  float m_run = kNegInf, l_run = 0.f;
  const size_t kv_stride = (size_t)a.s.hkv * D;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int ntiles = (it.nkv + KV_TILE - 1) / KV_TILE;
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    for (int e = tid; e < KV_TILE * D; e += T) {
      const int r = e / D, col = e % D;
      const int key = min(t * KV_TILE + r, it.nkv - 1);
      const size_t o2 = (size_t)kvl[key] * kv_stride + (size_t)hk * D + col;
      Kf[r * KP + col] = ((const float*)a.K)[o2];
      Vf[r * KP + col] = ((const float*)a.V)[o2];
    }
    __syncthreads();
    float s[KV_TILE];
    float mloc = kNegInf;
    for (int j = 0; j < KV_TILE; ++j) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < H; ++i) acc = fmaf(q[i], Kf[j * KP + half * H + i], acc);
      acc += __shfl_xor(acc, 1);
      const int kidx = t * KV_TILE + j;
      if (kidx >= it.nkv || it.kv_pos0 + kidx > qpos) acc = kNegInf;
      s[j] = acc * a.s.scale;
      mloc = fmaxf(mloc, s[j]);
    }
    const float m_new = fmaxf(m_run, mloc);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = expf(m_run - m_use);
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < H; ++i) o[i] *= alpha;
    for (int j = 0; j < KV_TILE; ++j) {
      const float p = expf(s[j] - m_use);
      l_run += p;
#pragma unroll
      for (int i = 0; i < H; ++i) o[i] = fmaf(p, Vf[j * KP + half * H + i], o[i]);
    }
    m_run = m_new;
  }
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  const float lse = l_run > 0.f ? m_run + logf(l_run) : kNegInf;
  if (!row_ok) return;
  float* op;
  if (it.part < 0) {
    op = (float*)a.O + ((size_t)row * a.s.hq + head) * D + half * H;
    if (half == 0) a.LSE[(size_t)head * a.s.ns + row] = lse;
  } else {
    const size_t prow = (size_t)it.part + ridx;
    op = a.part_o + (prow * a.s.hq + head) * D + half * H;
    if (half == 0) a.part_lse[prow * a.s.hq + head] = lse;
  }
#pragma unroll
  for (int i = 0; i < H; ++i) op[i] = o[i] * inv;
}

template <int D>
__global__ __launch_bounds__(256) void bwd_kv_f32_kernel(BwdArgs a) {
  constexpr int H = D / 2;
  constexpr int QP = D + 1;
  __shared__ float Qf[Q_SUB * QP];
  __shared__ float dOf[Q_SUB * QP];
  __shared__ float s_lse[Q_SUB], s_del[Q_SUB];
  __shared__ int s_qpos[Q_SUB];
  const BkvItem it = a.plan.bkv[blockIdx.x];
  const int tid = threadIdx.x;
  const int key = tid >> 1, half = tid & 1;
  const int hk = it.hk, G = a.s.g;
  const size_t kv_stride = (size_t)a.s.hkv * D;
  const int slot = a.plan.kv_list[it.kv_off + min(key, it.nk - 1)];
  const int kpos = it.kv_pos0 + key;
  float k[H], v[H], dk[H], dv[H];
  {
    const size_t o = (size_t)slot * kv_stride + (size_t)hk * D + half * H;
#pragma unroll
    for (int i = 0; i < H; ++i) {
      k[i] = ((const float*)a.K)[o + i];
      v[i] = ((const float*)a.V)[o + i];
      dk[i] = 0.f;
      dv[i] = 0.f;
    }
  }
  const int* ql = a.plan.q_list + it.q_off;
  const int nsub = (it.nq + Q_SUB - 1) / Q_SUB;
  for (int sub = 0; sub < nsub; ++sub)
    for (int g = 0; g < G; ++g) {
      const int head = hk * G + g;
      __syncthreads();
      for (int e = tid; e < Q_SUB * D; e += blockDim.x) {
        const int r = e / D, col = e % D;
        const int row = ql[min(Q_SUB * sub + r, it.nq - 1)];
        const size_t o = ((size_t)row * a.s.hq + head) * D + col;
        Qf[r * QP + col] = ((const float*)a.Q)[o];
        dOf[r * QP + col] = ((const float*)a.dO)[o];
      }
      if (tid < Q_SUB) {
        const int r = Q_SUB * sub + tid;
        const int row = ql[min(r, it.nq - 1)];
        s_lse[tid] = a.LSE[(size_t)head * a.s.ns + row];
        s_del[tid] = a.delta[(size_t)head * a.s.ns + row];
        s_qpos[tid] = r < it.nq ? a.plan.row_pos[row] : -1;
      }
      __syncthreads();
      for (int r = 0; r < Q_SUB; ++r) {
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int i = 0; i < H; ++i) {
          s = fmaf(Qf[r * QP + half * H + i], k[i], s);
          dp = fmaf(dOf[r * QP + half * H + i], v[i], dp);
        }
        s += __shfl_xor(s, 1);
        dp += __shfl_xor(dp, 1);
        float p = expf(s * a.s.scale - s_lse[r]);
        if (kpos > s_qpos[r]) p = 0.f;
        const float ds = p * (dp - s_del[r]);
#pragma unroll
        for (int i = 0; i < H; ++i) {
          dv[i] = fmaf(p, dOf[r * QP + half * H + i], dv[i]);
          dk[i] = fmaf(ds, Qf[r * QP + half * H + i], dk[i]);
        }
      }
    }
  if (key >= it.nk) return;
  float* kd;
  float* vd;
  if (it.part < 0) {
    const size_t o = (size_t)slot * kv_stride + (size_t)hk * D + half * H;
    kd = a.dK + o;
    vd = a.dV + o;
  } else {
    const size_t o = ((size_t)it.part * BKV_TILE + key) * D + half * H;
    kd = a.part_dk + o;
    vd = a.part_dv + o;
  }
#pragma unroll
  for (int i = 0; i < H; ++i) {
    kd[i] = dk[i] * a.s.scale;
    vd[i] = dv[i];
  }
}

template <int D>
__global__ __launch_bounds__(512) void bwd_dq_f32_kernel(BwdArgs a) {
  constexpr int H = D / 2;
  constexpr int KP = D + 1;
  __shared__ float Kf[KV_TILE * KP];
  __shared__ float Vf[KV_TILE * KP];
  const FwdItem it = a.plan.fwd[blockIdx.x];
  const int tid = threadIdx.x, T = blockDim.x;
  const int pair = tid >> 1, half = tid & 1;
  const int head = it.head0 + pair / a.s.bmq;
  const int hk = it.head0 / a.s.g;
  const int ridx = pair % a.s.bmq;
  const bool row_ok = ridx < it.nq;
  const int row = a.plan.q_list[it.q_off + (row_ok ? ridx : it.nq - 1)];
  const int qpos = a.plan.row_pos[row];
  const float lse = a.LSE[(size_t)head * a.s.ns + row];
  const float del = a.delta[(size_t)head * a.s.ns + row];
  float q[H], dov[H], dq[H];
  {
    const size_t o = ((size_t)row * a.s.hq + head) * D + half * H;
#pragma unroll
    for (int i = 0; i < H; ++i) {
      q[i] = ((const float*)a.Q)[o + i];
      dov[i] = ((const float*)a.dO)[o + i];
      dq[i] = 0.f;
    }
  }
  const size_t kv_stride = (size_t)a.s.hkv * D;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int ntiles = (it.nkv + KV_TILE - 1) / KV_TILE;
  for (int t = 0; t < ntiles; ++t) {
    __syncthreads();
    for (int e = tid; e < KV_TILE * D; e += T) {
      const int r = e / D, col = e % D;
      const int key = min(t * KV_TILE + r, it.nkv - 1);
      const size_t o2 = (size_t)kvl[key] * kv_stride + (size_t)hk * D + col;
      Kf[r * KP + col] = ((const float*)a.K)[o2];
      Vf[r * KP + col] = ((const float*)a.V)[o2];
    }
    __syncthreads();
    for (int j = 0; j < KV_TILE; ++j) {
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int i = 0; i < H; ++i) {
        s = fmaf(q[i], Kf[j * KP + half * H + i], s);
        dp = fmaf(dov[i], Vf[j * KP + half * H + i], dp);
      }
      s += __shfl_xor(s, 1);
      dp += __shfl_xor(dp, 1);
      const int kidx = t * KV_TILE + j;
      float p = expf(s * a.s.scale - lse);
      if (kidx >= it.nkv || it.kv_pos0 + kidx > qpos) p = 0.f;
      const float ds = p * (dp - del);
#pragma unroll
      for (int i = 0; i < H; ++i) dq[i] = fmaf(ds, Kf[j * KP + half * H + i], dq[i]);
    }
  }
  if (!row_ok) return;
  float* dst = it.part < 0 ? a.dQ + ((size_t)row * a.s.hq + head) * D + half * H
                           : a.part_dq + (((size_t)it.part + ridx) * a.s.hq + head) * D + half * H;
#pragma unroll
  for (int i = 0; i < H; ++i) dst[i] = dq[i] * a.s.scale;
}

// ============================================================================================
// Small row kernels (both dtypes)

// log-sum-exp merge of split forward pieces, fixed piece order
template <bool BF16>
__global__ __launch_bounds__(256) void fwd_merge_kernel(FwdArgs a) {
  const MergeEntry e = a.plan.merge[blockIdx.x];
  const int hq = a.s.hq, D = a.s.d, bmq = a.s.bmq;
  for (int idx = threadIdx.x; idx < e.nq * hq; idx += blockDim.x) {
    const int i = idx / hq, h = idx % hq;
    const int row = a.plan.q_list[e.q_off + i];
    float m = kNegInf;
    for (int j = 0; j < e.nparts; ++j) m = fmaxf(m, a.part_lse[((size_t)e.part0 + (size_t)j * bmq + i) * hq + h]);
    float wsum = 0.f;
    for (int j = 0; j < e.nparts; ++j) wsum += expf(a.part_lse[((size_t)e.part0 + (size_t)j * bmq + i) * hq + h] - m);
    const float lse = m + logf(wsum);
    a.LSE[(size_t)h * a.s.ns + row] = lse;
    for (int d4 = 0; d4 < D; d4 += 4) {
      f32x4 acc = f32x4{};
      for (int j = 0; j < e.nparts; ++j) {
        const size_t prow = (size_t)e.part0 + (size_t)j * bmq + i;
        const float w = expf(a.part_lse[prow * hq + h] - lse);
        const f32x4 x = *(const f32x4*)(a.part_o + (prow * hq + h) * D + d4);
        acc += w * x;
      }
      if (BF16) {
        u32x2 w2;
        w2[0] = pack2(acc[0], acc[1]);
        w2[1] = pack2(acc[2], acc[3]);
        *(u32x2*)((bf16_t*)a.O + ((size_t)row * hq + h) * D + d4) = w2;
      } else {
        *(f32x4*)((float*)a.O + ((size_t)row * hq + h) * D + d4) = acc;
      }
    }
  }
}

// Delta = rowsum(dO * O) per (row, head); D/8 lanes per (row, head), 8 elements each
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgs a) {
  const int D = a.s.d, hq = a.s.hq;
  const int lanes = D / 8;
  const int per_block = 256 / lanes;
  const int rh = blockIdx.x * per_block + threadIdx.x / lanes;
  const int sub = threadIdx.x % lanes;
  const bool ok = rh < a.s.ns * hq;
  float acc = 0.f;
  if (ok) {
    const size_t o = (size_t)rh * D + sub * 8;
    if (BF16) {
      const u32x4 x = ld16((const bf16_t*)a.O + o), y = ld16((const bf16_t*)a.dO + o);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc = fmaf(bf2f(x[e] & 0xffffu), bf2f(y[e] & 0xffffu), acc);
        acc = fmaf(bf2f(x[e] >> 16), bf2f(y[e] >> 16), acc);
      }
    } else {
      const float* x = (const float*)a.O + o;
      const float* y = (const float*)a.dO + o;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = fmaf(x[e], y[e], acc);
    }
  }
  for (int w = lanes / 2; w >= 1; w >>= 1) acc += __shfl_xor(acc, w);
  if (ok && sub == 0) {
    const int row = rh / hq, h = rh % hq;
    a.delta[(size_t)h * a.s.ns + row] = acc;
  }
}

// dK/dV = sum of partial tiles in ascending chunk order
__global__ __launch_bounds__(256) void bwd_reduce_kv_kernel(BwdArgs a) {
  const ReduceEntry e = a.plan.reduce[blockIdx.x];
  const int D = a.s.d;
  const size_t kv_stride = (size_t)a.s.hkv * D;
  for (int idx = threadIdx.x; idx < e.nk * (D / 4); idx += blockDim.x) {
    const int k = idx / (D / 4), d4 = (idx % (D / 4)) * 4;
    f32x4 sk = f32x4{}, sv = f32x4{};
    for (int j = 0; j < e.nparts; ++j) {
      const size_t o = (((size_t)e.part0 + j) * BKV_TILE + k) * D + d4;
      sk += *(const f32x4*)(a.part_dk + o);
      sv += *(const f32x4*)(a.part_dv + o);
    }
    const size_t o = (size_t)a.plan.kv_list[e.kv_off + k] * kv_stride + (size_t)e.hk * D + d4;
    *(f32x4*)(a.dK + o) = sk;
    *(f32x4*)(a.dV + o) = sv;
  }
}

// dQ = sum of partial rows in ascending piece order
__global__ __launch_bounds__(256) void bwd_reduce_dq_kernel(BwdArgs a) {
  const MergeEntry e = a.plan.merge[blockIdx.x];
  const int D = a.s.d, hq = a.s.hq, bmq = a.s.bmq;
  const int per_row = hq * D / 4;
  for (int idx = threadIdx.x; idx < e.nq * per_row; idx += blockDim.x) {
    const int i = idx / per_row, r = (idx % per_row) * 4;
    f32x4 acc = f32x4{};
    for (int j = 0; j < e.nparts; ++j)
      acc += *(const f32x4*)(a.part_dq + ((size_t)e.part0 + (size_t)j * bmq + i) * hq * D + r);
    const int row = a.plan.q_list[e.q_off + i];
    *(f32x4*)(a.dQ + (size_t)row * hq * D + r) = acc;
  }
}

// pool slots that hold no token get zero gradients
__global__ __launch_bounds__(256) void bwd_zero_pad_kernel(BwdArgs a) {
  const int per_slot = a.s.hkv * a.s.d / 4;
  const int64_t n = (int64_t)a.n_pad * per_slot;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * blockDim.x) {
    const int s = (int)(idx / per_slot), r = (int)(idx % per_slot) * 4;
    const size_t o = (size_t)a.plan.pad_slots[s] * a.s.hkv * a.s.d + r;
    *(f32x4*)(a.dK + o) = f32x4{};
    *(f32x4*)(a.dV + o) = f32x4{};
  }
}

}  // namespace

// ============================================================================================
// Launchers

#define PSATTN_NW_SWITCH(NW, BODY)                  \
  switch (NW) {                                     \
    case 4: { constexpr int W_ = 4; BODY; } break;  \
    case 5: { constexpr int W_ = 5; BODY; } break;  \
    case 6: { constexpr int W_ = 6; BODY; } break;  \
    case 7: { constexpr int W_ = 7; BODY; } break;  \
    case 8: { constexpr int W_ = 8; BODY; } break;  \
    default: return hipErrorInvalidValue;           \
  }

hipError_t launch_fwd_main(const FwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_items);
  if (bf16) {
    const dim3 block(a.s.nw * 64);
    if (a.s.d == 128) {
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((fwd_bf16_kernel<128, W_>), grid, block, 0, st, a));
    } else {
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((fwd_bf16_kernel<64, W_>), grid, block, 0, st, a));
    }
  } else {
    const dim3 block(2 * a.s.bmq * a.s.hc);  // two lanes per (row, head)
    if (a.s.d == 128) hipLaunchKernelGGL((fwd_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((fwd_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_fwd_merge(const FwdArgs& a, bool bf16, hipStream_t st) {
  if (bf16) hipLaunchKernelGGL((fwd_merge_kernel<true>), dim3(a.n_merge), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((fwd_merge_kernel<false>), dim3(a.n_merge), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16, hipStream_t st) {
  const int per_block = 256 / (a.s.d / 8);
  const int64_t n = (int64_t)a.s.ns * a.s.hq;
  const dim3 grid((unsigned)((n + per_block - 1) / per_block));
  if (bf16) hipLaunchKernelGGL((bwd_pre_kernel<true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((bwd_pre_kernel<false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_kv(const BwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_bkv), block(256);
  if (bf16) {
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_kv_bf16_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_kv_bf16_kernel<64>), grid, block, 0, st, a);
  } else {
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_kv_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_kv_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const BwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_fwd);
  if (bf16) {
    const dim3 block(a.s.nw * 64);
    if (a.s.d == 128) {
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((bwd_dq_bf16_kernel<128, W_>), grid, block, 0, st, a));
    } else {
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((bwd_dq_bf16_kernel<64, W_>), grid, block, 0, st, a));
    }
  } else {
    const dim3 block(2 * a.s.bmq * a.s.hc);
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_dq_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_dq_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_reduce_kv(const BwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(bwd_reduce_kv_kernel, dim3(a.n_reduce), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_reduce_dq(const BwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(bwd_reduce_dq_kernel, dim3(a.n_merge), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_zero_pad(const BwdArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.n_pad * a.s.hkv * a.s.d / 4;
  const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(bwd_zero_pad_kernel, dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace psattn
