// Forward kernels: bf16 MFMA main kernel, fp32 VALU kernel, log-sum-exp merge of split pieces.
//
// bf16 main kernel (gfx950).  One workgroup = one FwdItem: up to 32*rw query rows x hc query
// heads (all reading one kv head) x a range of keys along the node's root-to-node path.  Wave w
// owns head head0 + w / rw and 32 rows; it computes the transposed score tile S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16, so each lane holds one query row: softmax statistics are per-lane
// scalars and one v_permlane32_swap completes each row reduction.  The probabilities leave the
// accumulators as the B operand of O^T += V^T P^T without any data movement; V^T comes from a
// transposing LDS read (ds_read_b64_tr_b16) of the row-major V tile.
//
// Key tiles (64 keys) are gathered through the path's slot list, one 256-byte row per key and
// head, and copied global -> LDS directly (global_load_lds_dwordx4) into a two-stage ring; the
// copies for tile t+1 run while tile t is computed.  The running max is only moved when it grows
// by more than 2^8, so O and the row sum are rarely rescaled.
#include "psattn_device.h"

namespace psattn {
namespace {

using namespace dev;

template <int D, int NW, int NS>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int RB = D * 2;                      // bytes per tile row
  constexpr int CPR = D / 8;                     // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;                  // rows per 64-lane copy instruction
  constexpr int TB = KV_TILE * RB;               // bytes per K or V tile
  constexpr int NI = KV_TILE / RPI;              // copy instructions per tile and tensor
  constexpr int IPW = (NI + NW - 1) / NW;
  constexpr int KS = D / 16;                     // k-steps over head_dim
  constexpr int DB = D / 32;                     // 32-wide head_dim blocks of O
  constexpr int TPB = IDX_BLK / KV_TILE;         // key tiles per staged index block
  constexpr int CPW = 2 * (NI / NW);          // K+V copies every wave issues per tile (at least)
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NS][2][TB];   // [stage][K | V]
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
  const int nkv = it.nkv;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int ntiles = (nkv + KV_TILE - 1) / KV_TILE;

  if (tid < IDX_BLK) s_slot[0][tid] = kvl[min(tid, nkv - 1)];
  int pre = 0;
  if (tid < IDX_BLK && nkv > IDX_BLK) pre = kvl[min(IDX_BLK + tid, nkv - 1)];

  bf16x8 qreg[KS];
  {
    const bf16_t* qp = (const bf16_t*)a.Q + ((size_t)row * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) qreg[s] = as_bf(ld16(qp + 16 * s));
  }

  // LDS read offsets of this lane (independent of the tile and of the 32-row block)
  int koff[KS];          // row-major A operand: row l32, chunk 2s + hh
#pragma unroll
  for (int s = 0; s < KS; ++s) koff[s] = tile_off<D>(l32, 2 * s + hh);
  int voff[2][DB];       // transposing reads: rows 8rd + 4hh + r4, columns 32mb + dsub + 4j
  {
    const int r4 = (lane & 15) >> 2, j = lane & 3, dsub = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd)
#pragma unroll
      for (int mb = 0; mb < DB; ++mb)
        voff[rd][mb] = tile_off<D>(8 * rd + 4 * hh + r4, (32 * mb + dsub + 4 * j) >> 3) + 8 * (j & 1);
  }

  const size_t kv_stride = (size_t)a.s.hkv * D;
  const bf16_t* Kb = (const bf16_t*)a.K + (size_t)hk * D;
  const bf16_t* Vb = (const bf16_t*)a.V + (size_t)hk * D;
  const int crow = lane / CPR, cpc = lane % CPR;
  auto issue = [&](int t) {
    uint8_t* kdst = &smem[t % NS][0][0];
    uint8_t* vdst = &smem[t % NS][1][0];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
      const int k = wave + NW * i;
      if (NI % NW == 0 || k < NI) {
        const int r = k * RPI + crow;
        const int key = min(t * KV_TILE + r, nkv - 1);
        const int slot = s_slot[(key / IDX_BLK) & 1][key % IDX_BLK];
        const size_t go = (size_t)slot * kv_stride + ((cpc ^ swz<D>(r)) << 3);
        copy16_to_lds(Kb + go, kdst + k * 1024);
        copy16_to_lds(Vb + go, vdst + k * 1024);
      }
    }
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int mb = 0; mb < DB; ++mb) oacc[mb] = f32x16{};
  float m_run = kNegInf, l_run = 0.f;
  const float c = a.s.scale * kLog2e;
  const float th = 8.f / c;   // max growth (raw score units) tolerated before rescaling

  wait_vmem<0>();   // operands and index block loaded; nothing older stays in flight in the loop
  __syncthreads();
  // NS-stage ring: tiles t+1 .. t+NS-2 are in flight while tile t is computed.  Index blocks
  // (TPB tiles each) are double-buffered in LDS; block b+1 is fetched into registers when tile
  // TPB*b starts issuing and stored just before its first tile is issued.
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < ntiles) issue(p);
  for (int t = 0; t < ntiles; ++t) {
    const int tn = t + NS - 1;                 // tile issued in this iteration
    if (tn < ntiles && tn % TPB == 0 && tid < IDX_BLK) s_slot[(tn / TPB) & 1][tid] = pre;
    // this wave's copies for tile t are done once at most CPW*(NS-2) newer copies are in flight
    if (t + NS - 2 < ntiles) wait_vmem<CPW * (NS - 2)>();
    else wait_vmem<0>();
    __syncthreads();
    if (tn < ntiles) {
      issue(tn);
      if (tn % TPB == 0 && tid < IDX_BLK && (tn / TPB + 1) * IDX_BLK < nkv)
        pre = load_untracked(kvl + min((tn / TPB + 1) * IDX_BLK + tid, nkv - 1));
    }

    const uint8_t* Kt = &smem[t % NS][0][0];
    const uint8_t* Vt = &smem[t % NS][1][0];
    f32x16 sacc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      sacc[b] = f32x16{};
#pragma unroll
      for (int s = 0; s < KS; ++s) sacc[b] = mfma(as_bf(ld16(Kt + 32 * b * RB + koff[s])), qreg[s], sacc[b]);
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
    float mt = kNegInf;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[b][v]);
    mt = pair_max(mt);
    if (__any(mt > m_run + th)) {
      const float m_new = fmaxf(m_run, mt);
      const float alpha = m_new == kNegInf ? 1.f : fast_exp2((m_run - m_new) * c);
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < DB; ++mb) oacc[mb] *= alpha;
      m_run = m_new;
    }
    const float mc = m_run == kNegInf ? 0.f : m_run * c;
    float psum = 0.f;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = fast_exp2(fmaf(sacc[b][v], c, -mc));
        sacc[b][v] = p;
        psum += p;
      }
    l_run += psum;

    bf16x8 pb[2][2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      pb[b][0] = pack8(sacc[b], 0);
      pb[b][1] = pack8(sacc[b], 8);
    }
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
        for (int mb = 0; mb < DB; ++mb) {
          const uint8_t* vp = Vt + (32 * b + 16 * t2) * RB;
          oacc[mb] = mfma(as_bf(lds_tr(vp + voff[0][mb]), lds_tr(vp + voff[1][mb])), pb[b][t2], oacc[mb]);
        }
  }

  const float l_tot = pair_sum(l_run);
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

// ============================================================================================
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

}  // namespace

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
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((fwd_bf16_kernel<128, W_, 2>), grid, block, 0, st, a));
    } else {
      PSATTN_NW_SWITCH(a.s.nw, hipLaunchKernelGGL((fwd_bf16_kernel<64, W_, 2>), grid, block, 0, st, a));
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

}  // namespace psattn
