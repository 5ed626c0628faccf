// Forward kernels: bf16 MFMA main kernel, fp32 VALU kernel, log-sum-exp merge of split pieces.
//
// bf16 kernels (gfx950).  One workgroup = one FwdItem: 32*rw query rows x hc query heads (all
// reading one kv head) x a range of keys along the node's root-to-node path.  A wave computes the
// transposed score tile S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so each lane holds one query
// row: softmax statistics are per-lane scalars and one v_permlane32_swap completes each row
// reduction.  The probabilities leave the accumulators as the B operand of O^T += V^T P^T without
// any data movement; V^T comes from a transposing LDS read (ds_read_b64_tr_b16).
//
// Key tiles (64 keys) are gathered through the path's slot list, one row per key, and copied
// global -> LDS directly (global_load_lds_dwordx4) into a ring while earlier tiles are computed:
// a 4-stage ring in the grouped layout of gtile_off (fwd_bf16_w64_kernel, NH 32-row halves per
// wave).  The running max is only moved when it grows by more than 2^8, so O and the row sum
// are rarely rescaled.
#include "psattn_device.h"

#ifndef PSATTN_FWD_NS
#define PSATTN_FWD_NS 4
#endif
// 32-row halves per wavefront of the main bf16 kernel: 2 (one wavefront per SIMD) or 1 (two)
#ifndef PSATTN_FWD_NH
#define PSATTN_FWD_NH 1
#endif
// fragment prefetch distance of the main kernel, in MFMA pairs (6 measured best with two
// wavefronts per SIMD, within 256 registers)
#ifndef PSATTN_FWD_PF
#define PSATTN_FWD_PF (PSATTN_FWD_NH == 1 ? 6 : 4)
#endif

namespace psattn {
namespace {

using namespace dev;

// ============================================================================================
// bf16 main kernel.  A wavefront holds the queries (AGPRs), the output accumulators (AGPRs) and
// the scores (VGPRs) of NH 32-row halves of one head.  NH = 2: one wavefront per SIMD (up to 512
// registers), every K or V fragment read from LDS feeds two MFMAs.  NH = 1: eight wavefronts, two
// per SIMD (up to 256 registers each), so one wavefront's softmax issues while the other's MFMAs
// run, at twice the LDS reads per flop; measured the faster of the two on long prefixes.  Work
// proceeds in 32-key blocks j; stage j issues the score MFMAs of block j+1 and the PV MFMAs of
// block j-1, and between them the softmax of block j (its scores were finished during stage
// j-1).  The instruction order inside a stage is fixed (scheduling fences).  Key tiles (two
// blocks) come through an NS-stage LDS ring, one barrier per tile.
template <int D, int NW, int NS, int NH>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3 - NH, 3 - NH))) void fwd_bf16_w64_kernel(FwdArgs a) {
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;
  constexpr int RPI = 64 / CPR;
  constexpr int TB = KV_TILE * RB;
  constexpr int NI = KV_TILE / RPI;
  constexpr int IPW = NI / NW;
  constexpr int KS = D / 16;                     // score MFMAs per row half and block
  constexpr int DB = D / 32;
  constexpr int NPV = 2 * DB;                    // PV MFMAs per row half and block
  constexpr int TPB = IDX_BLK / KV_TILE;
  constexpr int CPW = 2 * IPW;                   // K+V copies every wave issues per tile
  static_assert(NI % NW == 0 && NS >= 3 && NS - 1 <= TPB, "tile copy split / ring depth");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NS][2][TB];
  __shared__ int s_slot[2][IDX_BLK];

  const FwdItem it = a.plan.fwd[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int rwn = a.s.rw / NH;                   // NH*32-row blocks per head
  const int head = it.head0 + wave / rwn;
  const int hk = it.head0 / a.s.g;
  const int nkv = it.nkv;
  const int* kvl = a.plan.kv_list + it.kv_off;
  const int ntiles = (nkv + KV_TILE - 1) / KV_TILE;

  for (int i = tid; i < IDX_BLK; i += NW * 64) {
    s_slot[0][i] = kvl[min(i, nkv - 1)];
    if (nkv > IDX_BLK) s_slot[1][i] = kvl[min(IDX_BLK + i, nkv - 1)];
  }

  int ridx[NH], row[NH], lim[NH];
  bool row_ok[NH];
  bf16x8 qreg[NH][KS];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    ridx[rh] = (wave % rwn) * (32 * NH) + 32 * rh + l32;
    row_ok[rh] = ridx[rh] < it.nq;
    row[rh] = a.plan.q_list[it.q_off + (row_ok[rh] ? ridx[rh] : it.nq - 1)];
    // key kidx of this item is visible to the row iff kidx <= lim
    lim[rh] = min(nkv - 1, a.plan.row_pos[row[rh]] - it.kv_pos0);
    const bf16_t* qp = (const bf16_t*)a.Q + ((size_t)row[rh] * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) qreg[rh][s] = as_bf(ld16(qp + 16 * s));
  }

  // LDS byte offsets of this lane's fragments inside a 32-key block (gtile_off layout):
  // K fragment s (rows l32, chunk 2s + hh) at koff[s & 1] + 1024 (s >> 1); V^T fragment of
  // k-step t2 and d block mb (rows 16 t2 + 8 rd + 4 hh + r4, chunks 4 mb + (dsub + 4 j) / 8) at
  // voff[rd] + 16 t2 RB + 1024 mb
  const int koff[2] = {gtile_off<D>(l32, hh), gtile_off<D>(l32, 2 + hh)};
  int voff[2];
  {
    const int r4 = (lane & 15) >> 2, j = lane & 3, dsub = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) voff[rd] = gtile_off<D>(8 * rd + 4 * hh + r4, (dsub + 4 * j) >> 3) + 8 * (j & 1);
  }
  static_assert(D == 128 || D == 64, "head_dim");
  static_assert(NW * NH == 8 && IPW * NW == CPR, "copies: NW / 4 waves per row group of a tile, IPW units each");

  // pool rows are addressed by 32-bit byte offsets from the head's base (the launcher checks that
  // the pools are under 4 GiB and 2^24 rows, so slot * kv_stride is one 24-bit multiply-add)
  const uint32_t kv_stride = (uint32_t)(a.s.hkv * D * sizeof(bf16_t));
  const uint8_t* Kb = (const uint8_t*)a.K + (size_t)hk * D * sizeof(bf16_t);
  const uint8_t* Vb = (const uint8_t*)a.V + (size_t)hk * D * sizeof(bf16_t);
  // Copies: row group cg = wave / (NW/4) (keys 16 cg .. 16 cg + 15) of every tile is filled by
  // NW/4 waves, wave w taking the IPW 1 KB units u0 + i, u0 = IPW (w mod NW/4), one per
  // instruction i (unit u holds chunks 4u .. 4u + 3).  Lane l writes chunk 4u + l / 16 of the
  // row at position l % 16, i.e. of key row (l % 16) ^ 4 (l / 16) of the group.
  const int cg = wave / (NW / 4), u0 = (wave % (NW / 4)) * IPW;
  const int crow = 16 * cg + ((lane & 15) ^ (4 * (lane >> 4)));
  const uint32_t cbyte = ((uint32_t)(lane >> 4) << 4) + 64 * u0;
  const uint32_t smem_base = lds_addr(&smem[0][0][0]) + cg * 16 * RB + u0 * 1024;
  // the slot of this lane's copy row in key tile t (the two staged index blocks are contiguous:
  // entry key sits at key mod 2*IDX_BLK)
  auto issue_slot = [&](int t) __attribute__((always_inline)) {
    const uint32_t key = (uint32_t)min(t * KV_TILE + crow, nkv - 1);
    return (&s_slot[0][0])[key & (2 * IDX_BLK - 1)];
  };
  // copy instruction i of a tile into ring slot rs, K (tensor 0) or V (tensor 1)
  auto issue_copy1 = [&](int rs, auto ic, int slot, int tensor) __attribute__((always_inline)) {
    constexpr int i = decltype(ic)::value;
    const uint32_t dst = smem_base + (uint32_t)((rs * 2 + tensor) * TB) + i * 1024;
    const uint32_t off = __umul24((uint32_t)slot, kv_stride) + cbyte;
    copy16_to_lds_off_imm<64 * i>(tensor ? Vb : Kb, off, dst);
  };
  // all copies into ring slot t % NS, of tile min(t, ntiles - 1): past the last tile a copy
  // refills a slot no one reads, so every iteration issues the same copies and waits the same
  auto issue = [&](int t) __attribute__((always_inline)) {
    const int slot = issue_slot(min(t, ntiles - 1));
    static_for<IPW>([&](auto ic) __attribute__((always_inline)) {
      issue_copy1(t % NS, ic, slot, 0);
      issue_copy1(t % NS, ic, slot, 1);
    });
  };
  auto fetch_index_block = [&](int b) __attribute__((always_inline)) {
    if (b * IDX_BLK >= nkv) return;
    for (int w = wave; w < IDX_BLK / 64; w += NW)
      copy4_to_lds(kvl + min(b * IDX_BLK + 64 * w + lane, nkv - 1), &s_slot[b & 1][64 * w]);
  };

  f32x16 oacc[NH][DB];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh)
#pragma unroll
    for (int mb = 0; mb < DB; ++mb) {
      oacc[rh][mb] = f32x16{};
      pin_a(oacc[rh][mb]);
    }
#pragma unroll
  for (int rh = 0; rh < NH; ++rh)
#pragma unroll
    for (int s = 0; s < KS; ++s) pin_a(qreg[rh][s]);
  valu_fence();
  float m_run[NH], l_run[NH];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    m_run[rh] = kNegInf;
    l_run[rh] = 0.f;
  }
  const float c = a.s.scale * kLog2e;
  const float th = 8.f / c;

  // ---- one stage.  Sc: scores of block j (softmax now, K rows at Kc); Sn: scores of block
  // j+1 (MFMAs now, K rows at Kn); Pp: probabilities of block j-1 (PV MFMAs now, V rows at Vp);
  // Pc: block j's probabilities (written).  extra(IntC<i>) runs after MFMA slot i.
  //
  // The softmax exponentiates against the running max of the earlier blocks while block j's
  // own row max is reduced alongside, so no exponential waits for a reduction.  A row whose max
  // grows by more than 2^8 (always the case for the first block of a row) sends the whole wave
  // down a slow path after the stage: block j's scores are recomputed from Kc, exponentiated
  // against the new max, and O and the running sum are rescaled.
  auto scores = [&](const uint8_t* Kb_, f32x16 (&S)[NH]) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 k = as_bf(ld16(Kb_ + koff[s & 1] + (s >> 1) * 1024));
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) {
        if (s == 0) mma_v_first(S[rh], k, qreg[rh][s]);
        else mma_v(S[rh], k, qreg[rh][s]);
      }
    }
  };
  auto mask_elem = [&](f32x16 (&S)[NH], int rh, int v, int kb) __attribute__((always_inline)) {
    // element v holds key kb + 4*hh + 8*(v/4) + v%4, visible iff it is <= lim
    const int x = lim[rh] - kb - 4 * hh;
    S[rh][v] = (8 * (v >> 2) + (v & 3) > x) ? kNegInf : S[rh][v];
  };
  auto stage = [&](f32x16 (&Sc)[NH], f32x16 (&Sn)[NH], const bf16x8 (&Pp)[NH][2], bf16x8 (&Pc)[NH][2],
                   const uint8_t* Kc, const uint8_t* Kn, const uint8_t* Vp, int kb, auto masked,
                   auto extra, auto pv_first) __attribute__((always_inline)) {
    float mx[NH], mt[NH], ps[NH][2], l_prev[NH], mc[NH];
    bool g[NH];
#pragma unroll
    for (int rh = 0; rh < NH; ++rh) mc[rh] = m_run[rh] == kNegInf ? 0.f : m_run[rh] * c;
    // element e = 16 rh + v is scaled at chunk F(e), exponentiated at F(e)+1, summed at F(e)+2
    auto F = [](int e) constexpr { return (e * 29) / (16 * NH); };
    auto chunk = [&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      if constexpr (q == 0) {
#pragma unroll
        for (int rh = 0; rh < NH; ++rh) l_prev[rh] = l_run[rh];
      }
      if constexpr (q < 8) {          // mask, then row max steps over elements 2q, 2q+1 of both halves
#pragma unroll
        for (int rh = 0; rh < NH; ++rh) {
          if constexpr (decltype(masked)::value) {
            mask_elem(Sc, rh, 2 * q, kb);
            mask_elem(Sc, rh, 2 * q + 1, kb);
          }
          if constexpr (q == 0) mx[rh] = max2f(Sc[rh][0], Sc[rh][1]);
          else mx[rh] = max3f(mx[rh], Sc[rh][2 * q], Sc[rh][2 * q + 1]);
          anchor(mx[rh]);
        }
      }
      if constexpr (q == 9) {
#pragma unroll
        for (int rh = 0; rh < NH; ++rh) {
          mt[rh] = pair_max2(mx[rh]);
          anchor(mt[rh]);
        }
      }
      if constexpr (q == 11) {
#pragma unroll
        for (int rh = 0; rh < NH; ++rh) g[rh] = mt[rh] > m_run[rh] + th;
      }
      static_for<16 * NH>([&](auto ec) __attribute__((always_inline)) {
        constexpr int e = decltype(ec)::value, rh = e / 16, v = e % 16;
        if constexpr (F(e) == q) Sc[rh][v] = fmaf(Sc[rh][v], c, -mc[rh]);
        if constexpr (F(e) + 1 == q) Sc[rh][v] = fast_exp2(Sc[rh][v]);
        if constexpr (F(e) + 2 == q) {
          if constexpr (v < 2) ps[rh][v] = Sc[rh][v];
          else ps[rh][v & 1] += Sc[rh][v];
          anchor(ps[rh][v & 1]);
        }
        if constexpr (v % 8 == 7 && F(e) + 2 == q) {
          Pc[rh][v / 8] = pack8(Sc[rh], 8 * (v / 8));
          anchor(Pc[rh][v / 8]);
        }
      });
      if constexpr (q == 31) {
#pragma unroll
        for (int rh = 0; rh < NH; ++rh) {
          l_run[rh] += ps[rh][0] + ps[rh][1];
          anchor(l_run[rh]);
        }
      }
    };
    static_assert(F(16 * NH - 1) + 2 <= 31, "softmax schedule");
    bf16x8 kf[KS], vf[NPV];
    auto load_k = [&](int s) __attribute__((always_inline)) { kf[s] = as_bf(ld16(Kn + koff[s & 1] + (s >> 1) * 1024)); };
    auto load_v = [&](int u) __attribute__((always_inline)) {   // u = DB * t2 + mb
      const int t2 = u / DB, mb = u % DB;
      const int o = 16 * t2 * RB + 1024 * mb;
      vf[u] = as_bf(lds_tr(Vp + voff[0] + o), lds_tr(Vp + voff[1] + o));
    };
    // fragments in use order (K fragments then V fragments, or V first when pv_first); each is
    // read PF MFMA pairs ahead of the pair that consumes it
    constexpr bool PVF = decltype(pv_first)::value;
    constexpr int PF = PSATTN_FWD_PF;
    auto load_frag = [&](int f) __attribute__((always_inline)) {
      if (PVF) {
        if (f < NPV) load_v(f);
        else if (f < NPV + KS) load_k(f - NPV);
      } else {
        if (f < KS) load_k(f);
        else if (f < KS + NPV) load_v(f - KS);
      }
    };
#pragma unroll
    for (int f = 0; f < PF; ++f) load_frag(f);
    constexpr int NSLOT = NH * KS + NH * NPV;
    auto slot = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      constexpr int iq = PVF ? (i >= NH * NPV ? i - NH * NPV : -1) : (i < NH * KS ? i : -1);   // score slot index
      constexpr int ip = PVF ? (i < NH * NPV ? i : -1) : (i >= NH * KS ? i - NH * KS : -1);    // PV slot index
      if constexpr (iq >= 0) {
        constexpr int s = iq / NH, rh = iq % NH;
        if constexpr (rh == 0) load_frag((PVF ? NPV : 0) + s + PF);
        if constexpr (s == 0) mma_v_first(Sn[rh], kf[s], qreg[rh][s]);
        else mma_v(Sn[rh], kf[s], qreg[rh][s]);
      } else {
        constexpr int u = ip / NH, rh = ip % NH;
        constexpr int t2 = u / DB, mb = u % DB;
        if constexpr (rh == 0) load_frag((PVF ? 0 : KS) + u + PF);
        mma_a(oacc[rh][mb], vf[u], Pp[rh][t2]);
      }
      // softmax chunks [32 i / NSLOT, 32 (i+1) / NSLOT) follow slot i
      static_for<(32 * (i + 1)) / NSLOT - (32 * i) / NSLOT>([&](auto dq) __attribute__((always_inline)) {
        chunk(IntC<(32 * i) / NSLOT + decltype(dq)::value>{});
      });
      extra(ic);
      sched_fence();
    };
    static_for<NSLOT>(slot);
    bool gany = g[0];
#pragma unroll
    for (int rh = 1; rh < NH; ++rh) gany = gany || g[rh];
    if (__any(gany)) {
      // slow path: new row maxima.  Recompute block j's scores (its K rows are still resident),
      // exponentiate them against the new maxima, and rescale O and the running sums.
      f32x16 R[NH];
      scores(Kc, R);
      mfma_fence();
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) {
        pin_v(R[rh]);
        const float m_new = g[rh] ? mt[rh] : m_run[rh];
        const float alpha = (g[rh] && m_run[rh] != kNegInf) ? fast_exp2((m_run[rh] - m_new) * c) : 1.f;
        m_run[rh] = m_new;
        const float mcn = m_new == kNegInf ? 0.f : m_new * c;
        float sum = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          if constexpr (decltype(masked)::value) mask_elem(R, rh, v, kb);
          R[rh][v] = fast_exp2(fmaf(R[rh][v], c, -mcn));
          sum += R[rh][v];
        }
        l_run[rh] = l_prev[rh] * alpha + sum;
        Pc[rh][0] = pack8(R[rh], 0);
        Pc[rh][1] = pack8(R[rh], 8);
#pragma unroll
        for (int mb = 0; mb < DB; ++mb) {
          pin_a(oacc[rh][mb]);
          oacc[rh][mb] *= alpha;
        }
      }
    }
  };
  wait_vmem<0>();
  __syncthreads();
#pragma unroll
  for (int p = 0; p < NS - 1; ++p) issue(p);
  wait_vmem<CPW * (NS - 2)>();
  __syncthreads();

  f32x16 SA[NH], SB[NH];
  bf16x8 PA[NH][2], PB[NH][2];
  // block 0's scores; block -1's probabilities are zero (its PV products, on tile 0's V rows,
  // add nothing)
  scores(&smem[0][0][0], SA);
#pragma unroll
  for (int rh = 0; rh < NH; ++rh)
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) PB[rh][t2] = bf16x8{};
  mfma_fence();

  auto tile = [&](int t, auto masked) __attribute__((always_inline)) {
    const uint8_t* Kt = &smem[t % NS][0][0];
    const uint8_t* Vt = &smem[t % NS][1][0];
    const uint8_t* Vprev = t > 0 ? &smem[(t + NS - 1) % NS][1][0] + 32 * RB : Vt;
    const int tn = t + NS - 1;
    const int slot = issue_slot(min(tn, ntiles - 1));
    // stage 2t: scores of block 2t+1, PV of block 2t-1, softmax of block 2t; K copies
    auto kcopies = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i % 4 == 2 && i / 4 < IPW) issue_copy1(tn % NS, IntC<i / 4>{}, slot, 0);
    };
    stage(SA, SB, PB, PA, Kt, Kt + 32 * RB, Vprev, t * KV_TILE, masked, kcopies, Flag<false>{});
    // tile t+1 must be resident before its first block's scores: newer copies are K and V of
    // tiles t+2 .. t+NS-2 and K of tile t+NS-1
    wait_vmem<(2 * NS - 5) * IPW>();
    __syncthreads();
    // stage 2t+1: PV of block 2t first (V rows resident before the barrier), then the scores of
    // block 2t+2 (K rows of tile t+1; unused past the last tile), softmax of 2t+1; V copies
    auto vcopies = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i % 4 == 2 && i / 4 < IPW) issue_copy1(tn % NS, IntC<i / 4>{}, slot, 1);
      if constexpr (i == 4 * IPW + 2) {
        if (tn < ntiles && tn % TPB == 0 && tn >= TPB) fetch_index_block(tn / TPB + 1);
      }
    };
    stage(SB, SA, PA, PB, Kt + 32 * RB, &smem[(t + 1) % NS][0][0], Vt, t * KV_TILE + 32, masked, vcopies, Flag<true>{});
  };
  int t = 0;
  for (; t < min(it.nfull, ntiles); ++t) tile(t, Flag<false>{});
  for (; t < ntiles; ++t) tile(t, Flag<true>{});
  wait_vmem<0>();   // no copy may still be writing this workgroup's LDS when it ends
  // PV of the last block
  {
    const uint8_t* Vl = &smem[(ntiles - 1) % NS][1][0] + 32 * RB;
#pragma unroll
    for (int u = 0; u < NPV; ++u) {
      const int t2 = u / DB, mb = u % DB;
      const int o = 16 * t2 * RB + 1024 * mb;
      const bf16x8 v = as_bf(lds_tr(Vl + voff[0] + o), lds_tr(Vl + voff[1] + o));
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) mma_a(oacc[rh][mb], v, PB[rh][t2]);
    }
    mfma_fence();
#pragma unroll
    for (int rh = 0; rh < NH; ++rh)
#pragma unroll
      for (int mb = 0; mb < DB; ++mb) pin_a(oacc[rh][mb]);
  }

  // Unsplit items write O as whole rows: each wave stages its normalized bf16 rows in the LDS ring
  // (free once every wave has finished the PV products above; padded row stride OS), then copies
  // them out 16 bytes per lane, 1 KB of consecutive row bytes per instruction.  Row index and
  // validity of staged row r come from lane r % 32 of the half that owns it.  With O_lo, a second
  // pass stages and writes the rounding residuals O - bf16(O) the same way.
  constexpr int OS = RB + 16;
  static_assert(NW * 32 * NH * OS <= NS * 2 * TB, "staged O rows fit the ring");
  const bool direct = it.part < 0;
  uint8_t* ot = &smem[0][0][0] + wave * (32 * NH) * OS;
  float inv[NH];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    const float l_tot = pair_sum(l_run[rh]);
    inv[rh] = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float lse = l_tot > 0.f ? m_run[rh] * a.s.scale + logf(l_tot) : kNegInf;
    if (direct) {
      if (row_ok[rh] && hh == 0) a.LSE[(size_t)head * a.s.ns + row[rh]] = lse;
      continue;
    }
    if (!row_ok[rh]) continue;
    {
      const size_t prow = (size_t)it.part + ridx[rh];
      float* op = a.part_o + (prow * a.s.hq + head) * D;
#pragma unroll
      for (int mb = 0; mb < DB; ++mb)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          *(f32x4*)(op + 32 * mb + 8 * g4 + 4 * hh) =
              f32x4{oacc[rh][mb][4 * g4] * inv[rh], oacc[rh][mb][4 * g4 + 1] * inv[rh], oacc[rh][mb][4 * g4 + 2] * inv[rh],
                    oacc[rh][mb][4 * g4 + 3] * inv[rh]};
      if (hh == 0) a.part_lse[prow * a.s.hq + head] = lse;
    }
  }
  if (direct) {
    // first pass: bf16(O) into O; second pass: bf16(O - bf16(O)) into O_lo
    auto write_rows = [&](bool lo, uint8_t* dst) __attribute__((always_inline)) {
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) {
        uint8_t* orow = ot + (32 * rh + l32) * OS;
#pragma unroll
        for (int mb = 0; mb < DB; ++mb)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x[e] = oacc[rh][mb][4 * g4 + e] * inv[rh];
              if (lo) x[e] -= bf2f(pack2(x[e], 0.f) & 0xffffu);
            }
            u32x2 w;
            w[0] = pack2(x[0], x[1]);
            w[1] = pack2(x[2], x[3]);
            *(u32x2*)(orow + 2 * (32 * mb + 8 * g4 + 4 * hh)) = w;
          }
      }
      constexpr int CPRO = RB / 16, RPIO = 64 / CPRO;   // 16-byte chunks per row, rows per instruction
      const int ch = lane % CPRO;
#pragma unroll
      for (int k = 0; k < 32 * NH / RPIO; ++k) {
        const int rl = k * RPIO + lane / CPRO;          // staged row; its half is (k * RPIO) / 32
        const int rh = (k * RPIO) / 32;
        const int r = __shfl(row[rh], rl % 32);
        const int ok = __shfl((int)row_ok[rh], rl % 32);
        const u32x4 v = *(const u32x4*)(ot + rl * OS + 16 * ch);
        if (ok) *(u32x4*)(dst + ((size_t)r * a.s.hq + head) * RB + 16 * ch) = v;
      }
    };
    __syncthreads();
    write_rows(false, (uint8_t*)a.O);
    // (the staging area is the wave's own: its LDS reads above complete before the writes below)
    if (a.O_lo) write_rows(true, (uint8_t*)a.O_lo);
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
  // D/4 lanes per (row, head), 4 elements each (coalesced rows); blockIdx.y slices the pairs
  const MergeEntry e = a.plan.merge[blockIdx.x];
  const int hq = a.s.hq, D = a.s.d, bmq = a.s.bmq;
  const int lanes = D / 4, per_pass = 256 / lanes;
  const int d4 = 4 * (threadIdx.x % lanes);
  for (int pr = blockIdx.y * per_pass + threadIdx.x / lanes; pr < e.nq * hq; pr += gridDim.y * per_pass) {
    const int i = pr / hq, h = pr % hq;
    const int row = a.plan.q_list[e.q_off + i];
    float m = kNegInf;
    for (int j = 0; j < e.nparts; ++j) m = fmaxf(m, a.part_lse[((size_t)e.part0 + (size_t)j * bmq + i) * hq + h]);
    float wsum = 0.f;
    for (int j = 0; j < e.nparts; ++j) wsum += expf(a.part_lse[((size_t)e.part0 + (size_t)j * bmq + i) * hq + h] - m);
    const float lse = m + logf(wsum);
    if (d4 == 0) a.LSE[(size_t)h * a.s.ns + row] = lse;
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
      if (a.O_lo) {
        u32x2 r2;
        r2[0] = pack2(acc[0] - bf2f(w2[0] & 0xffffu), acc[1] - bf2f(w2[0] >> 16));
        r2[1] = pack2(acc[2] - bf2f(w2[1] & 0xffffu), acc[3] - bf2f(w2[1] >> 16));
        *(u32x2*)((bf16_t*)a.O_lo + ((size_t)row * hq + h) * D + d4) = r2;
      }
    } else {
      *(f32x4*)((float*)a.O + ((size_t)row * hq + h) * D + d4) = acc;
    }
  }
}

}  // namespace

hipError_t launch_fwd_main(const FwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_items);
  if (bf16) {
    // 8 / NH waves of NH*32 rows (the planner makes every item 8 (subtile, head) pairs); the pools
    // are addressed by 32-bit byte offsets (the host rejects larger trees)
    if (a.s.rw % PSATTN_FWD_NH != 0 || a.s.nw != 8) return hipErrorInvalidValue;
    const dim3 block(8 / PSATTN_FWD_NH * 64);
    if (a.s.d == 128) hipLaunchKernelGGL((fwd_bf16_w64_kernel<128, 8 / PSATTN_FWD_NH, PSATTN_FWD_NS, PSATTN_FWD_NH>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((fwd_bf16_w64_kernel<64, 8 / PSATTN_FWD_NH, PSATTN_FWD_NS, PSATTN_FWD_NH>), grid, block, 0, st, a);
  } else {
    const dim3 block(2 * a.s.bmq * a.s.hc);  // two lanes per (row, head)
    if (a.s.d == 128) hipLaunchKernelGGL((fwd_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((fwd_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_fwd_merge(const FwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_merge, kMergeSlices);
  if (bf16) hipLaunchKernelGGL((fwd_merge_kernel<true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((fwd_merge_kernel<false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace psattn
