// Backward kernels: Delta = rowsum(dO * O), dK/dV (keys stationary), dQ (queries stationary),
// fixed-order reductions of split partial results, and zeroing of pool slots holding no token.
//
// bf16 dK/dV kernel (gfx950).  One workgroup = one BkvItem: up to 128 keys of one node and one
// kv head (wave w keeps keys 32w..32w+31 of K and V in registers) x a chunk of the rows that
// consume them -- the node's own later rows and every row of every descendant node, i.e. all
// branches reusing the prefix.  For each 32-row subtile and each query head of the group it
// computes S = Q K^T and dP = dO V^T (lane <-> key), P = exp(S*scale - LSE), dS = P*(dP - Delta),
// then dV += P^T dO and dK += dS^T Q, whose B operands (dO^T, Q^T) come from transposing LDS
// reads of the row-major tiles.  Q/dO tiles and the LSE/Delta rows are copied global -> LDS
// directly into a two-stage ring.  Consumer-row indices are staged in LDS 256 at a time.
//
// bf16 dQ kernel: same items and wave layout as the forward kernel; recomputes S^T and dP^T per
// key tile and accumulates dQ^T += K^T dS^T, K^T again from transposing reads.
#include <algorithm>

#include "psattn_device.h"

namespace psattn {
namespace {

using namespace dev;

template <int D>
__global__ __launch_bounds__(256) void bwd_kv_bf16_kernel(BwdArgs a) {
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;
  constexpr int RPI = 64 / CPR;
  constexpr int QB = Q_SUB * RB;              // bytes per Q or dO subtile
  constexpr int NI = Q_SUB / RPI;             // copy instructions per subtile and tensor
  constexpr int IPW = NI / 4;                 // per wave
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int SPB = IDX_BLK / Q_SUB;        // subtiles per staged row block
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2][2][QB];   // [stage][Q | dO]
  __shared__ __attribute__((aligned(16))) float s_stat[2][2][Q_SUB];  // [stage][LSE | Delta][row]
  __shared__ int s_row[2][IDX_BLK];
  __shared__ int s_qpos[2][IDX_BLK];
  __shared__ int s_slot[BKV_TILE];

  const BkvItem it = a.plan.bkv[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int hk = it.hk, G = a.s.g, hq = a.s.hq, ns = a.s.ns;
  const int nq = it.nq;
  const int* ql = a.plan.q_list + it.q_off;
  const size_t kv_stride = (size_t)a.s.hkv * D;

  if (tid < BKV_TILE) s_slot[tid] = a.plan.kv_list[it.kv_off + min(tid, it.nk - 1)];
  {
    const int r = ql[min(tid, nq - 1)];
    s_row[0][tid] = r;
    s_qpos[0][tid] = tid < nq ? a.plan.row_pos[r] : -1;
  }
  int pre_row = 0, pre_qpos = -1;
  if (nq > IDX_BLK) {
    pre_row = ql[min(IDX_BLK + tid, nq - 1)];
    pre_qpos = IDX_BLK + tid < nq ? a.plan.row_pos[pre_row] : -1;
  }

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
  int koff[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) koff[s] = tile_off<D>(l32, 2 * s + hh);
  int voff[2][DB];
  {
    const int r4 = (lane & 15) >> 2, j = lane & 3, dsub = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd)
#pragma unroll
      for (int nb = 0; nb < DB; ++nb)
        voff[rd][nb] = tile_off<D>(8 * rd + 4 * hh + r4, (32 * nb + dsub + 4 * j) >> 3) + 8 * (j & 1);
  }

  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int nb = 0; nb < DB; ++nb) {
    dk[nb] = f32x16{};
    dv[nb] = f32x16{};
  }

  const int nsub = (nq + Q_SUB - 1) / Q_SUB;
  const int nsteps = nsub * G;
  const int crow = lane / CPR, cpc = lane % CPR;
  auto issue = [&](int step) {
    const int st = step & 1, sub = step / G, head = hk * G + step % G;
    const int* rows = &s_row[(sub / SPB) & 1][(sub % SPB) * Q_SUB];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int k = wave + 4 * i;
      const int r = k * RPI + crow;
      const size_t go = ((size_t)rows[r] * hq + head) * D + ((cpc ^ swz<D>(r)) << 3);
      copy16_to_lds((const bf16_t*)a.Q + go, &smem[st][0][k * 1024]);
      copy16_to_lds((const bf16_t*)a.dO + go, &smem[st][1][k * 1024]);
    }
    if (lane < 16) {
      const int r = 16 * (wave & 1) + lane;
      const float* src = (wave >> 1) ? a.delta : a.LSE;
      copy4_to_lds(src + (size_t)head * ns + rows[r], &s_stat[st][wave >> 1][16 * (wave & 1)]);
    }
  };

  const float c = a.s.scale * kLog2e;
  wait_vmem<0>();   // operands and index block loaded; nothing older stays in flight in the loop
  __syncthreads();
  issue(0);
  for (int step = 0; step < nsteps; ++step) {
    const int sn = step + 1;
    const bool new_blk = sn < nsteps && sn % G == 0 && (sn / G) % SPB == 0;
    if (new_blk) {
      const int blk = (sn / G) / SPB;
      s_row[blk & 1][tid] = pre_row;
      s_qpos[blk & 1][tid] = pre_qpos;
    }
    wait_vmem<0>();
    __syncthreads();
    if (sn < nsteps) {
      issue(sn);
      if (new_blk) {
        const int nxt = ((sn / G) / SPB + 1) * IDX_BLK + tid;
        if (nxt - tid < nq) {
          pre_row = ql[min(nxt, nq - 1)];
          pre_qpos = nxt < nq ? a.plan.row_pos[pre_row] : -1;
        }
      }
    }

    const int st = step & 1, sub = step / G;
    const uint8_t* Qt = &smem[st][0][0];
    const uint8_t* dOt = &smem[st][1][0];
    f32x16 S = f32x16{}, dP = f32x16{};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      S = mfma(as_bf(ld16(Qt + koff[s])), kreg[s], S);
      dP = mfma(as_bf(ld16(dOt + koff[s])), vreg[s], dP);
    }
    // accumulator layout: lane <-> key (column l32), element v <-> row 8*(v/4) + 4*hh + v%4
    const bool need_mask = (Q_SUB * sub < it.nmask) || (Q_SUB * sub + Q_SUB > nq);
    const int* qp = &s_qpos[(sub / SPB) & 1][(sub % SPB) * Q_SUB];
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 L = *(const f32x4*)&s_stat[st][0][8 * g4 + 4 * hh];
      const f32x4 Dl = *(const f32x4*)&s_stat[st][1][8 * g4 + 4 * hh];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 4 * g4 + e;
        float p = fast_exp2(fmaf(S[v], c, -L[e] * kLog2e));
        if (need_mask && kpos > qp[8 * g4 + 4 * hh + e]) p = 0.f;
        S[v] = p;
        dP[v] = p * (dP[v] - Dl[e]);
      }
    }
    const bf16x8 pa0 = pack8(S, 0), pa1 = pack8(S, 8);
    const bf16x8 sa0 = pack8(dP, 0), sa1 = pack8(dP, 8);
#pragma unroll
    for (int nb = 0; nb < DB; ++nb) {
      dv[nb] = mfma(pa0, as_bf(lds_tr(dOt + voff[0][nb]), lds_tr(dOt + voff[1][nb])), dv[nb]);
      dv[nb] = mfma(pa1, as_bf(lds_tr(dOt + 16 * RB + voff[0][nb]), lds_tr(dOt + 16 * RB + voff[1][nb])), dv[nb]);
      dk[nb] = mfma(sa0, as_bf(lds_tr(Qt + voff[0][nb]), lds_tr(Qt + voff[1][nb])), dk[nb]);
      dk[nb] = mfma(sa1, as_bf(lds_tr(Qt + 16 * RB + voff[0][nb]), lds_tr(Qt + 16 * RB + voff[1][nb])), dk[nb]);
    }
  }

  // accumulator layout: lane <-> head_dim column 32*nb + l32, element v <-> key of this wave
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

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void bwd_dq_bf16_kernel(BwdArgs a) {
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;
  constexpr int RPI = 64 / CPR;
  constexpr int TB = KV_TILE * RB;
  constexpr int NI = KV_TILE / RPI;
  constexpr int IPW = (NI + NW - 1) / NW;
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int TPB = IDX_BLK / KV_TILE;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2][2][TB];   // [stage][K | V]
  __shared__ int s_slot[2][IDX_BLK];

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
  const int nkv = it.nkv;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int ntiles = (nkv + KV_TILE - 1) / KV_TILE;

  if (tid < IDX_BLK) s_slot[0][tid] = kvl[min(tid, nkv - 1)];
  int pre = 0;
  if (tid < IDX_BLK && nkv > IDX_BLK) pre = kvl[min(IDX_BLK + tid, nkv - 1)];

  bf16x8 qreg[KS], doreg[KS];
  {
    const size_t o = ((size_t)row * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qreg[s] = as_bf(ld16((const bf16_t*)a.Q + o + 16 * s));
      doreg[s] = as_bf(ld16((const bf16_t*)a.dO + o + 16 * s));
    }
  }
  int koff[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) koff[s] = tile_off<D>(l32, 2 * s + hh);
  int toff[2][DB];
  {
    const int r4 = (lane & 15) >> 2, j = lane & 3, dsub = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd)
#pragma unroll
      for (int mb = 0; mb < DB; ++mb)
        toff[rd][mb] = tile_off<D>(8 * rd + 4 * hh + r4, (32 * mb + dsub + 4 * j) >> 3) + 8 * (j & 1);
  }

  const size_t kv_stride = (size_t)a.s.hkv * D;
  const bf16_t* Kb = (const bf16_t*)a.K + (size_t)hk * D;
  const bf16_t* Vb = (const bf16_t*)a.V + (size_t)hk * D;
  const int crow = lane / CPR, cpc = lane % CPR;
  auto issue = [&](int t) {
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int k = wave + NW * i;
      if (NI % NW == 0 || k < NI) {
        const int r = k * RPI + crow;
        const int key = min(t * KV_TILE + r, nkv - 1);
        const int slot = s_slot[(key / IDX_BLK) & 1][key % IDX_BLK];
        const size_t go = (size_t)slot * kv_stride + ((cpc ^ swz<D>(r)) << 3);
        copy16_to_lds(Kb + go, &smem[t & 1][0][k * 1024]);
        copy16_to_lds(Vb + go, &smem[t & 1][1][k * 1024]);
      }
    }
  };

  f32x16 dq[DB];
#pragma unroll
  for (int mb = 0; mb < DB; ++mb) dq[mb] = f32x16{};
  const float c = a.s.scale * kLog2e;

  wait_vmem<0>();   // operands and index block loaded; nothing older stays in flight in the loop
  __syncthreads();
  issue(0);
  for (int t = 0; t < ntiles; ++t) {
    const int tn = t + 1;
    if (tn < ntiles && tn % TPB == 0 && tid < IDX_BLK) s_slot[(tn / TPB) & 1][tid] = pre;
    wait_vmem<0>();
    __syncthreads();
    if (tn < ntiles) {
      issue(tn);
      if (tn % TPB == 0 && tid < IDX_BLK && (tn / TPB + 1) * IDX_BLK < nkv)
        pre = kvl[min((tn / TPB + 1) * IDX_BLK + tid, nkv - 1)];
    }

    const uint8_t* Kt = &smem[t & 1][0][0];
    const uint8_t* Vt = &smem[t & 1][1][0];
    f32x16 S[2], dP[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      S[b] = f32x16{};
      dP[b] = f32x16{};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        S[b] = mfma(as_bf(ld16(Kt + 32 * b * RB + koff[s])), qreg[s], S[b]);
        dP[b] = mfma(as_bf(ld16(Vt + 32 * b * RB + koff[s])), doreg[s], dP[b]);
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
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int mb = 0; mb < DB; ++mb) {
          const uint8_t* kp = Kt + (32 * b + 16 * t2) * RB;
          dq[mb] = mfma(as_bf(lds_tr(kp + toff[0][mb]), lds_tr(kp + toff[1][mb])), sb[b][t2], dq[mb]);
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
// fp32 path (VALU).

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

#define PSATTN_NW_SWITCH(NW, BODY)                  \
  switch (NW) {                                     \
    case 5: { constexpr int W_ = 5; BODY; } break;  \
    case 6: { constexpr int W_ = 6; BODY; } break;  \
    case 7: { constexpr int W_ = 7; BODY; } break;  \
    case 8: { constexpr int W_ = 8; BODY; } break;  \
    default: return hipErrorInvalidValue;           \
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
