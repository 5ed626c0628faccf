// Backward kernels: Delta = rowsum(dO * O), dK/dV (keys stationary), dQ (queries stationary),
// fixed-order reductions of split partial results, and zeroing of pool slots holding no token.
//
// bf16 dK/dV kernel (gfx950).  One workgroup = one BkvItem: up to 128 keys of one node and one
// kv head x a chunk of the rows that consume them -- the node's own later rows and every row of
// every descendant node, i.e. all branches reusing the prefix.  For each 32-row subtile and each
// query head of the group it computes S = Q K^T and dP = dO V^T (lane <-> key),
// P = exp(S*scale - LSE), dS = P*(dP - Delta), then dV += P^T dO and dK += dS^T Q, whose B
// operands (dO^T, Q^T) come from transposing LDS reads of the row-major tiles.  The kernel
// (bwd_kv_bf16_1w_kernel) runs one wavefront per SIMD, wave w keeping keys 32w..32w+31 of K and
// V and their dK/dV accumulators in registers, and streams Q/dO rows and the LSE/Delta values
// global -> LDS directly into a five-step ring.  Consumer-row indices and positions are staged
// in LDS 256 at a time, each block copied there (LDS-DMA) two iterations before it is read.
//
// bf16 dQ kernel: the same items as the forward kernel and its structure (NH 32-row halves per
// wave); recomputes S^T and dP^T per key tile and accumulates dQ^T += K^T dS^T, K^T again from
// transposing reads.
#include <algorithm>

#include "psattn_device.h"

// 32-row halves per wavefront of the bf16 dQ kernel: 2 (one wavefront per SIMD) or 1 (two; with
// Q, dO and dQ in 128 AGPRs it has 128 VGPRs for the rest, and measured 1-3% slower on a
// 32q/8kv-head, d = 128 tree of a 4096-token prefix and 16 branches of 1024)
#ifndef PSATTN_DQ_NH
#define PSATTN_DQ_NH 2
#endif
// fragment prefetch distance of the dQ kernel (3 keeps the two-wavefront form within 128 VGPRs)
#ifndef PSATTN_DQ_PF
#define PSATTN_DQ_PF (PSATTN_DQ_NH == 1 ? 3 : 4)
#endif

// Remainder products in the dK/dV kernel on steps with large P or dS (1); 0 rounds P and dS once
// everywhere (a timing variant: its error grows with the number of consumers of a key)
#ifndef PSATTN_KV_REM
#define PSATTN_KV_REM 1
#endif

namespace psattn {
namespace {

using namespace dev;

// ============================================================================================
// bf16 dK/dV kernel, one wavefront per SIMD.  Four wavefronts: wave w owns keys 32w .. 32w+31
// of the tile for every query head; its K and V rows (the B operands of S = Q K^T and
// dP = dO V^T) and its dK and dV accumulators stay in AGPRs for the whole item.  The consumer
// rows stream through LDS one step at a time (a step is a 32-row subtile of one query head:
// Q, dO and their LSE log2 e and Delta), in a five-deep ring.  Iteration i issues the dV/dK
// MFMAs of step i-1 (dV += P^T dO, dK += dS^T Q), then the S and dP MFMAs of step i+1, and
// between them computes P = exp2(S c - LSE log2 e) and dS = P (dP - Delta) of step i.
template <int D, bool REM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void bwd_kv_bf16_1w_kernel(BwdArgs a) {
  constexpr int RB = D * 2;
  constexpr int LRB = D == 128 ? 8 : 7;       // log2(RB)
  constexpr int CPR = D / 8;
  constexpr int RPI = 64 / CPR;
  constexpr int QB = Q_SUB * RB;              // bytes per Q or dO subtile of one head
  constexpr int NI = Q_SUB / RPI;             // copy instructions per subtile and tensor
  constexpr int KS = D / 16, DB = D / 32;
  constexpr int SPB = IDX_BLK / Q_SUB;        // subtiles per staged row block
  constexpr int NR = 5;                       // step ring: steps i-1 .. i+NR-2 (copied NR-2 ahead)
  constexpr int CPS = 2 * NI / 4;             // copies every wave issues per step (Q and dO)
  static_assert((2 * NI) % 4 == 0 && (1 << LRB) == RB, "copy split");
  static_assert(SPB > NR + 1, "the first NR steps read row block 0; a buffer is refilled after its readers");
  constexpr int PER = NR % 2 == 0 ? NR : 2 * NR;   // loop trip: the S/dP buffers alternate with period 2
  static_assert(2 * SPB == 16 && IDX_BLK == SPB * Q_SUB, "subtile sub is staged at entry (sub & 15) * Q_SUB");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NR][2][QB];   // [step slot][Q | dO]
  __shared__ __attribute__((aligned(16))) uint32_t s_stat[NR][Q_SUB][2];  // [step slot][row][-LSE/scale | -Delta] as (hi, lo) bf16
  __shared__ int s_row[2][IDX_BLK];
  __shared__ int s_qpos[2][IDX_BLK];
  const uint32_t smem_base = lds_addr(&smem[0][0][0]), stat_base = lds_addr(&s_stat[0][0][0]);

  const BkvItem it = a.plan.bkv[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int hk = it.hk, G = a.s.g, hq = a.s.hq, ns = a.s.ns;
  const int nq = it.nq;
  const int* ql = a.plan.q_list + it.q_off;
  const int crow = lane / CPR, cpc = lane % CPR;
  const uint32_t kv_stride = (uint32_t)(a.s.hkv * D * sizeof(bf16_t));

  // consumer rows staged 256 at a time: row index (past the list: the last row again) and
  // sequence position (past the list: -1, the q_pos entry before the array).  Block 0 here; block
  // B >= 1 by LDS-DMA two iterations before its first copy step (see the iteration)
  const int* qp = a.plan.q_pos + it.q_off;
  s_row[0][tid] = ql[min(tid, nq - 1)];
  s_qpos[0][tid] = tid < nq ? qp[tid] : -1;
  auto stage_block = [&](int blk) __attribute__((always_inline)) {
    const int e = blk * IDX_BLK + tid;
    copy4_to_lds(ql + min(e, nq - 1), &s_row[blk & 1][64 * wave]);
    copy4_to_lds(e < nq ? qp + e : a.plan.q_pos - 1, &s_qpos[blk & 1][64 * wave]);
  };
  // K and V rows of this wave's keys: B operands (lane <-> key, 8 consecutive head_dim entries
  // per k-slot)
  bf16x8 kreg[KS], vreg[KS];
  {
    const int key = min(32 * wave + l32, it.nk - 1);
    const size_t o = (size_t)__umul24((uint32_t)a.plan.kv_list[it.kv_off + key], kv_stride) +
                     (size_t)hk * D * sizeof(bf16_t) + 16 * hh;
    const uint8_t* kp = (const uint8_t*)a.K + o;
    const uint8_t* vp = (const uint8_t*)a.V + o;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      kreg[s] = as_bf(ld16(kp + 32 * s));
      vreg[s] = as_bf(ld16(vp + 32 * s));
    }
  }
  const int kpos = it.kv_pos0 + 32 * wave + l32;
  f32x16 dk[DB], dv[DB];
#pragma unroll
  for (int nb = 0; nb < DB; ++nb) {
    dk[nb] = f32x16{};
    dv[nb] = f32x16{};
    pin_a(dk[nb]);
    pin_a(dv[nb]);
  }
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    pin_a(kreg[s]);
    pin_a(vreg[s]);
  }
  valu_fence();

  const int nsub = (nq + Q_SUB - 1) / Q_SUB;
  const int nsteps = nsub * G;                // step = subtile * G + head
  // ---- copies.  Copy instruction j of this wave moves 16 bytes per lane of row r_j = ins*RPI + crow
  // of a subtile of tensor tens (Q or dO); its source byte offset is the lane's rowoff_j (row of the
  // list times hq*RB, plus the swizzled column: changes with the subtile) plus hoff = (hk*G + h)*RB
  // (uniform: changes with the head).  Every wave also copies the step's -LSE/scale (even lanes)
  // and -Delta (odd lanes) of its 32 rows, the same 256 bytes, so that all waves issue and wait
  // alike.
  struct Rows {
    uint32_t off[CPS];   // rowoff_j
    uint32_t st;         // 4 * row lane/2 (+ the distance from the -LSE/scale to the -Delta array on odd lanes)
  };
  const uint32_t nd_dist = (uint32_t)((const char*)a.kv_nd - (const char*)a.kv_nls);
  const uint32_t stat_row = (uint32_t)hq * 4;   // bytes per row of the [Ns][Hq] statistics
  const uint32_t row_bytes = (uint32_t)hq * RB;
  // rows of subtile sub (staged): the LDS reads, then the offsets (split, so that the reads can be
  // issued well before their results are needed)
  struct RowIdx {
    int r[CPS + 1];
  };
  auto read_rows = [&](int sub) __attribute__((always_inline)) {
    const int* rows = &s_row[0][0] + (sub & 15) * Q_SUB;
    RowIdx x;
#pragma unroll
    for (int j = 0; j < CPS; ++j) x.r[j] = rows[((wave + 4 * j) % NI) * RPI + crow];
    x.r[CPS] = rows[lane >> 1];
    return x;
  };
  auto row_offsets = [&](const RowIdx& x) __attribute__((always_inline)) {
    Rows o;
#pragma unroll
    for (int j = 0; j < CPS; ++j) {
      const int r = ((wave + 4 * j) % NI) * RPI + crow;
      o.off[j] = (uint32_t)x.r[j] * row_bytes + ((cpc ^ swz<D>(r)) << 4);
    }
    o.st = (uint32_t)x.r[CPS] * stat_row + ((lane & 1) ? nd_dist : 0u);
    return o;
  };
  auto fetch_rows = [&](int sub) __attribute__((always_inline)) { return row_offsets(read_rows(sub)); };
  const void* gsrc[CPS];                      // tensor of copy j
  uint32_t gdst[CPS];                         // its LDS byte offset within a ring slot
#pragma unroll
  for (int j = 0; j < CPS; ++j) {
    const int k = wave + 4 * j, tens = k / NI, ins = k % NI;
    gsrc[j] = tens ? a.dO : a.Q;
    gdst[j] = (uint32_t)(tens * QB + ins * 1024);
  }
  const uint32_t hoff0 = (uint32_t)(hk * G) * RB, hst0 = (uint32_t)(hk * G) * 4;
  // copy j of a step (head offsets hoff/hst, ring slot byte offset slot_off) into its ring slot
  auto issue_one = [&](uint32_t slot_off, uint32_t hoff, const Rows& rw, int j) __attribute__((always_inline)) {
    copy16_to_lds_off(gsrc[j], rw.off[j] + hoff, smem_base + slot_off + gdst[j]);
  };
  auto issue_stat = [&](uint32_t slot_off, uint32_t hst, const Rows& rw) __attribute__((always_inline)) {
    copy4_to_lds_off(a.kv_nls, rw.st + hst, stat_base + slot_off / (2 * QB) * (2 * Q_SUB * 4));
  };

  const float c = a.s.scale * kLog2e;
  const int arow = l32 * RB, asw = swz<D>(l32);
  const int r4 = (lane & 15) >> 2, jq = lane & 3, dsub = 16 * ((lane >> 4) & 1);
  const int tcol = (dsub + 4 * jq) >> 3, tbyte = 8 * (jq & 1);
  const int trow0 = (4 * hh + r4) * RB, tsw0 = swz<D>(4 * hh + r4);
  const int trow1 = (8 + 4 * hh + r4) * RB, tsw1 = swz<D>(8 + 4 * hh + r4);
  // this lane's byte offsets, within a Q or dO subtile, of its fragment reads: computed once, so
  // that a read address is one add of the (uniform) subtile offset
  uint32_t aoff[KS], toff0[DB], toff1[DB];
#pragma unroll
  for (int s = 0; s < KS; ++s) aoff[s] = arow + (((2 * s + hh) ^ asw) << 4);
#pragma unroll
  for (int nb = 0; nb < DB; ++nb) {
    toff0[nb] = trow0 + (((4 * nb + tcol) ^ tsw0) << 4) + tbyte;
    toff1[nb] = trow1 + (((4 * nb + tcol) ^ tsw1) << 4) + tbyte;
  }
  const uint8_t* const sm = &smem[0][0][0];
  // base: byte offset of a subtile in smem
  auto ld_a = [&](uint32_t base, int s) __attribute__((always_inline)) { return as_bf(ld16(sm + (base + aoff[s]))); };
  auto ld_t = [&](uint32_t base, int u) __attribute__((always_inline)) {   // u = DB * t2 + nb
    const int t2 = u / DB, nb = u % DB;
    const uint32_t b = base + 16 * t2 * RB;
    return as_bf(lds_tr(sm + (b + toff0[nb])), lds_tr(sm + (b + toff1[nb])));
  };

  // steps whose rows may see only part of the tile ([mask_lo, mask_hi) of the list) or lie past
  // the list lie in [s_lo, s_hi) or [s_pad, nsteps); the mask is applied from the first of them on
  // (on a step whose rows see every key it changes nothing)
  const int s_lo = it.mask_lo / Q_SUB * G, s_hi = (it.mask_hi + Q_SUB - 1) / Q_SUB * G;
  const int s_pad = nq / Q_SUB * G;
  const int s_mask = s_lo < s_hi ? min(s_lo, s_pad) : s_pad;

  // ---- iteration i, NSLOT MFMA slots in NP pairs:
  //   pairs 0 .. NT-1: dV[nb] += P^T dO and dK[nb] += dS^T Q of step i-1 (pair u = DB*t2 + nb)
  //   (REM) then, on a step where some P > 2^-9 or |dS| > 2^-5: the same products of the
  //         remainders P - bf16(P) and dS - bf16(dS), from step i-1's fp32 P and dS
  //   pair NT:         S and dP of step i+1 start as -LSE/scale and -Delta (the statistics pair)
  //   then:            S += Q K^T and dP += dO V^T of step i+1 (pair = k-step s)
  // with P and dS of step i computed between them.  Sc/dPc: step i; Sn/dPn: step i+1 (written
  // from pair NT on; until then they still hold step i-1's fp32 P and dS); Pp/Sp: packed P and dS
  // of step i-1; Pc/Sc2: of step i (written).  S and dP thus leave the MFMAs as S - LSE/scale and
  // dP - Delta: P = exp2(c S') and dS = P dP' take two VALU products.
  // Why the remainders: dV_j = sum_i P_ij dO_i sums over every consumer of key j.  A single bf16
  // rounding of P leaves up to 2^-8 relative error per term, and these errors add up like a random
  // walk, ~2^-8/sqrt(3) * sqrt(sum_i P_ij^2 dO_i^2) at most: on a key that many consumers weight
  // heavily (a shared prefix token with attention-sink-like scores) that grows without bound.
  // With P = hi + lo, both bf16, each term is good to ~2^-16.  A step is left single-rounded only
  // when all its P <= 2^-9 (each term then off by <= 2^-17) and all |dS| <= 2^-5 (<= 2^-13); the
  // same holds for dS in dK = dS^T Q.  The forward and dQ products sum over keys, whose weights
  // P_i. add up to 1, and need no remainder terms.
  constexpr int NT = 2 * DB;                  // dV/dK slot pairs
  constexpr int PF = 3;
  constexpr int NP = NT + 1 + KS;             // pairs: dV/dK, statistics, S/dP k-steps
  constexpr int NSLOT = 2 * NP;
  constexpr int BAR = 2 * (NT - PF) - 1 < 3 ? 2 * (NT - PF) - 1 : 3;
  constexpr int CP0 = BAR + 1, CPD = 3;       // copy j of step i+3 at slot CP0 + CPD*j
  constexpr int ST_SLOT = CP0 + CPD * CPS, ROW_SLOT = ST_SLOT + 2;
  static_assert(BAR >= 1 && ROW_SLOT < NSLOT && 2 * (NT - PF) > BAR && ROW_SLOT > BAR + 1, "iteration schedule");
  static_assert(SPB > NR, "the first row block staged in the loop is staged at iteration >= 0");
  bf16x8 ftv[NT], ftk[NT];                    // transposed dO and Q fragments of the dV/dK pairs
  Rows rows_nx;                               // row offsets of the copy step's subtile
  // The statistics pair: S and dP of a step start as MFMAs of A = (hi, lo) of the row's -LSE/scale
  // and (hi, lo) of its -Delta, each split into two bf16 (relative error 2^-16), in k = 0..3, with
  // B = (1, 1, 0, 0, ...) or (0, 0, 1, 1, 0, ...) on every key: one 64-bit LDS read per lane
  // instead of 32 values.  B is zero on lanes 32-63 (k = 8..15), where A repeats the row's pairs.
  bf16x8 bs1 = as_bf(hh ? u32x4{0u, 0u, 0u, 0u} : u32x4{0x3F803F80u, 0u, 0u, 0u});
  bf16x8 bd1 = as_bf(hh ? u32x4{0u, 0u, 0u, 0u} : u32x4{0u, 0x3F803F80u, 0u, 0u});
  pin_a(bs1);
  pin_a(bd1);
  auto ld_stat = [&](uint32_t slot_off) __attribute__((always_inline)) {
    const uint32_t* st = &s_stat[0][0][0] + slot_off / (2 * QB) * (2 * Q_SUB);
    const u32x2 x = ld8(st + 2 * l32);
    return as_bf(u32x4{x[0], x[1], 0u, 0u});
  };
  // the causal mask, on a step whose rows may see only part of the tile (or lie past the list,
  // position -1): S of a hidden (row, key) pair becomes -inf before its exponential.  Every
  // other step skips it.
  auto mask_s = [&](f32x16& S, int step, int sub) __attribute__((always_inline)) {   // sub: step's subtile
    if (step >= s_mask) {
      mfma_fence();   // S was written by MFMAs of the previous iteration
      const int* qpp = &s_qpos[0][0] + (sub & 15) * Q_SUB;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int4 q = *(const int4*)&qpp[8 * g + 4 * hh];
#pragma unroll
        for (int k = 0; k < 4; ++k) S[4 * g + k] = kpos > q[k] ? kNegInf : S[4 * g + k];
      }
    }
  };
  // remainder products of one step, if any of its P > 2^-9 or |dS| > 2^-5 (wave-uniform branch):
  // Pf/Sf its fp32 P and dS, Ph/Sh their packed bf16, Qs/dOs its ring slot.  The maxima are
  // eight steps each: step k of the P maximum takes elements {0, 1, 2}, then {2k+1, 2k+2}, then
  // {15}; step k of the |dS| maximum takes {2k, 2k+1}.
  constexpr float kRemP = 1.0f / 512, kRemS = 1.0f / 32;
  auto max_p_step = [&](float& mp, const f32x16& Pf, int k) __attribute__((always_inline)) {
    if (k == 0) mp = max3f(Pf[0], Pf[1], Pf[2]);
    else if (k < 7) mp = max3f(mp, Pf[2 * k + 1], Pf[2 * k + 2]);
    else mp = max2f(mp, Pf[15]);
  };
  auto max_s_step = [&](float& ms, const f32x16& Sf, int k) __attribute__((always_inline)) {
    ms = max3abs(k == 0 ? 0.f : ms, Sf[2 * k], Sf[2 * k + 1]);
  };
  auto rem_apply = [&](float mp, float ms, const f32x16& Pf, const f32x16& Sf, const bf16x8 (&Ph)[2],
                       const bf16x8 (&Sh)[2], uint32_t Qs, uint32_t dOs) __attribute__((always_inline)) {
    if (__builtin_amdgcn_ballot_w64(mp > kRemP || ms > kRemS) == 0) return;
    bf16x8 pl[2], sl[2];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      pl[t2] = pack8_rem(Pf, 8 * t2, Ph[t2]);
      sl[t2] = pack8_rem(Sf, 8 * t2, Sh[t2]);
      anchor(pl[t2]);   // written before the fence, not next to an MFMA
      anchor(sl[t2]);
    }
    valu_fence();
#pragma unroll
    for (int u = 0; u < NT; ++u) {
      const int t2 = u / DB, nb = u % DB;
      mma_a(dv[nb], pl[t2], ld_t(dOs, u));
      mma_a(dk[nb], sl[t2], ld_t(Qs, u));
    }
  };
  auto remainders = [&](const f32x16& Pf, const f32x16& Sf, const bf16x8 (&Ph)[2], const bf16x8 (&Sh)[2], uint32_t Qs,
                        uint32_t dOs) __attribute__((always_inline)) {
    float mp = 0.f, ms = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      max_p_step(mp, Pf, k);
      max_s_step(ms, Sf, k);
    }
    rem_apply(mp, ms, Pf, Sf, Ph, Sh, Qs, dOs);
  };
  int h3, subc;                               // head of the copy step i+3 and subtile of min(i+3, nsteps-1)
  // row block staging: block stage_blk is staged in the iteration where to_stage reaches 0
  int stage_blk = 1, to_stage = SPB * G - NR;
  int h0 = 0, sub0 = 0;                       // head and subtile of step i
  uint32_t hoff3, hst3;                       // its head offsets in Q/dO rows and in the statistics
  auto body = [&](f32x16& Sc, f32x16& dPc, f32x16& Sn, f32x16& dPn, const bf16x8 (&Pp)[2], const bf16x8 (&Sp)[2],
                  bf16x8 (&Pc)[2], bf16x8 (&Sc2)[2], int i, auto pos) __attribute__((always_inline)) {
    // pos = i mod PER: the ring slots of steps i-1, i, i+1 and i+NR-2 are compile-time constants, so
    // that a read address is an immediate offset from the lane's base (step -1 reads ring slot
    // NR-1, zero-filled before the loop, with zero P and dS)
    constexpr int p = decltype(pos)::value;
    constexpr uint32_t Qp = (uint32_t)((p + NR - 1) % NR) * 2 * QB, dOp = Qp + QB;
    constexpr uint32_t Qc = (uint32_t)(p % NR) * 2 * QB, dOc = Qc + QB;
    constexpr uint32_t Qn = (uint32_t)((p + 1) % NR) * 2 * QB, dOn = Qn + QB;
    constexpr uint32_t slot3 = (uint32_t)((p + NR - 2) % NR) * 2 * QB;
    const bool next_sub = i + NR - 1 < nsteps && h3 == G - 1;   // step i+4 starts a subtile
    const bool new_blk = next_sub && (subc + 1) % SPB == 0;      // ... and a row block
    RowIdx rows_raw;
    bf16x8 fq[KS], fo[KS], ast;
    auto load_frag = [&](int f) __attribute__((always_inline)) {   // operands of pair f
      // (the operand of the pair's second MFMA is read first: the wait for the first covers both)
      if (f < NT) {
        ftk[f] = ld_t(Qp, f);
        ftv[f] = ld_t(dOp, f);
      } else if (f == NT) {
        ast = ld_stat(Qn);
      } else if (f <= NT + KS) {
        fo[f - NT - 1] = ld_a(dOn, f - NT - 1);
        fq[f - NT - 1] = ld_a(Qn, f - NT - 1);
      } else if (f < NP + PF) {
        ftk[f - NP] = ld_t(Qc, f - NP);
        ftv[f - NP] = ld_t(dOc, f - NP);
      }
    };
    // element v of this step's 16 per lane: scaled at F(v), exponentiated at F(v)+2 (a slot of
    // other work between the product and the exponential that reads it, so that no wait states are
    // padded), dS at F(v)+3; each 8-element half packed after its last one
    constexpr auto F = [](int v) { return 2 + (v * (NSLOT - 8)) / 16; };
    static_assert(F(15) + 4 < NSLOT, "P and dS packed within the iteration");
    auto chunk = [&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      static_for<16>([&](auto vc) __attribute__((always_inline)) {
        constexpr int v = decltype(vc)::value;
        // (each result pinned to its slot: the branches of the iteration would otherwise let the
        // compiler sink these products to their first use)
        if constexpr (F(v) == q) {
          float t = Sc[v] * c;
          anchor(t);
          Sc[v] = t;
        }
        if constexpr (F(v) + 2 == q) {
          float t = fast_exp2(Sc[v]);
          anchor(t);
          Sc[v] = t;
        }
        if constexpr (F(v) + 3 == q) {
          float t = Sc[v] * dPc[v];
          anchor(t);
          dPc[v] = t;
        }
        if constexpr (v % 8 == 7 && F(v) + 4 == q) {
          Pc[v / 8] = pack8(Sc, 8 * (v / 8));
          Sc2[v / 8] = pack8(dPc, 8 * (v / 8));
          anchor(Pc[v / 8]);
          anchor(Sc2[v / 8]);
        }

      });
    };
    // the remainder test of step i-1 runs alongside its dV/dK pairs: the maxima of its fp32 P (in
    // Sn) and dS (in dPn) take one step per MFMA slot, the P maximum after the dV MFMAs and the
    // |dS| maximum after the dK MFMAs; the ballot and the remainder products follow the last pair
    float rem_p = 0.f, rem_s = 0.f;
    auto slot = [&](auto ic) __attribute__((always_inline)) {
      constexpr int si = decltype(ic)::value;
      constexpr int m = si / 2, w = si % 2;
      if constexpr (si == 0) mask_s(Sc, i, sub0);
      if constexpr (REM && si == 2 * NT) {   // before the statistics pair overwrites Sn / dPn
        rem_apply(rem_p, rem_s, Sn, dPn, Pp, Sp, Qp, dOp);
        sched_fence();
      }
      if constexpr (w == 0) load_frag(m + PF);
      if constexpr (m < NT) {
        constexpr int t2 = m / DB, nb = m % DB;
        if constexpr (w == 0) mma_a(dv[nb], Pp[t2], ftv[m]);
        else mma_a(dk[nb], Sp[t2], ftk[m]);
      } else if constexpr (m == NT) {
        if constexpr (w == 0) mma_v_first(Sn, ast, bs1);
        else mma_v_first(dPn, ast, bd1);
      } else {
        constexpr int s = m - NT - 1;
        if constexpr (w == 0) mma_v(Sn, fq[s], kreg[s]);
        else mma_v(dPn, fo[s], vreg[s]);
      }
      chunk(ic);
      if constexpr (REM && m < NT) {
        static_for<8 / NT + (8 % NT ? 1 : 0)>([&](auto jc) __attribute__((always_inline)) {
          constexpr int k = m * 8 / NT + decltype(jc)::value;
          if constexpr (k < (m + 1) * 8 / NT) {
            if constexpr (w == 0) {
              max_p_step(rem_p, Sn, k);
              anchor(rem_p);
            } else {
              max_s_step(rem_s, dPn, k);
              anchor(rem_s);
            }
          }
        });
      }
      if constexpr (si == BAR) {
        // (a row block staged by LDS-DMA two iterations ago is older than the last iteration's
        // copies: this wait covers it, and the barrier makes it visible)
        wait_vmem<(NR - 4) * (CPS + 1)>();
        barrier_only();
      }
      if constexpr (si == BAR + 1) {
        if (next_sub) rows_raw = read_rows(subc + 1);
      }
      if constexpr (si >= CP0 && si < CP0 + CPD * CPS && (si - CP0) % CPD == 0) issue_one(slot3, hoff3, rows_nx, (si - CP0) / CPD);
      if constexpr (si == ST_SLOT) issue_stat(slot3, hst3, rows_nx);
      if constexpr (si == ROW_SLOT) {
        if (next_sub) {
          subc += 1;
          rows_nx = row_offsets(rows_raw);
        }
        // row block stage_blk starts at step stage_blk * SPB * G, the copy step of iteration i + 3,
        // and iteration i + 2 reads its first subtile's rows: stage it now (the copies of
        // iteration i + 1 then lie between it and that read's wait), into the buffer of block
        // stage_blk - 2, whose last reader was more than SPB * G - 6 steps ago
        if (--to_stage == 0) {
          if (stage_blk * IDX_BLK < nq) stage_block(stage_blk);
          stage_blk += 1;
          to_stage = SPB * G;
        }
      }
      sched_fence();
    };
    static_for<NSLOT>(slot);
    {
      const bool wrap = h0 == G - 1;
      h0 = wrap ? 0 : h0 + 1;
      sub0 += wrap ? 1 : 0;
    }
    // the copy step's head advances (past the last step the rows stay those of the last subtile,
    // so any head still addresses rows of the list)
    {
      const bool wrap = h3 == G - 1;
      h3 = wrap ? 0 : h3 + 1;
      hoff3 = wrap ? hoff0 : hoff3 + RB;
      hst3 = wrap ? hst0 : hst3 + 4;
    }
  };

  // ring slot NR-1 (read as step -1 by iteration 0) zero-filled
  for (int k = tid; k < 2 * QB / 16; k += 256) *(u32x4*)&smem[NR - 1][0][16 * k] = u32x4{0, 0, 0, 0};
  wait_vmem<0>();   // K and V registers, index block
  __syncthreads();
#pragma unroll
  for (int p = 0; p < NR - 2; ++p) {
    const int sc = min(p, nsteps - 1), h = sc % G;
    const Rows rw = fetch_rows(sc / G);
#pragma unroll
    for (int j = 0; j < CPS; ++j) issue_one(p * 2 * QB, hoff0 + h * RB, rw, j);
    issue_stat(p * 2 * QB, hst0 + (uint32_t)h * 4, rw);
  }
  {
    const int sc = min(NR - 2, nsteps - 1);
    h3 = sc % G;
    subc = sc / G;
    hoff3 = hoff0 + h3 * RB;
    hst3 = hst0 + (uint32_t)h3 * 4;
    rows_nx = fetch_rows(subc);
  }
  wait_vmem<(NR - 3) * (CPS + 1)>();
  __syncthreads();

  f32x16 SA, SB, dPA, dPB;
  bf16x8 PA[2], PB[2], DSA[2], DSB[2];
  // S and dP of step 0; the P and dS of step -1 are zero (its dV/dK products, on step 0's rows,
  // add nothing); the first dV/dK fragments of iteration 0 (step 0's rows)
  {
    const uint32_t Q0 = 0, dO0 = QB;
    bf16x8 a0 = ld_stat(0);
    anchor(a0);
    valu_fence();
    mma_v_first(SA, a0, bs1);
    mma_v_first(dPA, a0, bd1);
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      mma_v(SA, ld_a(Q0, s), kreg[s]);
      mma_v(dPA, ld_a(dO0, s), vreg[s]);
    }
#pragma unroll
    for (int f = 0; f < PF; ++f) {
      ftv[f] = ld_t(dO0, f);
      ftk[f] = ld_t(Q0, f);
    }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      PB[t2] = DSB[t2] = bf16x8{};
      anchor(PB[t2]);   // the zeros are written here, before the fence, not next to an MFMA
      anchor(DSB[t2]);
    }
    // step -1's fp32 P and dS (read by iteration 0's remainder test) are zero
    SB = dPB = f32x16{};
    anchor(SB);
    anchor(dPB);
    mfma_fence();
  }

  // PER iterations per trip (the S/dP buffers alternate with period 2, the ring with period NR),
  // leaving after whichever iteration is the last
  int i = 0;
  for (;;) {
    bool done = false;
    static_for<PER>([&](auto pc) __attribute__((always_inline)) {
      constexpr int p = decltype(pc)::value;
      if (!done) {
        if constexpr (p % 2 == 0) body(SA, dPA, SB, dPB, PB, DSB, PA, DSA, i, pc);
        else body(SB, dPB, SA, dPA, PA, DSA, PB, DSB, i, pc);
        done = ++i == nsteps;
      }
    });
    if (done) break;
  }
  // the S and dP of step nsteps (never used) are still being written: keep their registers
  // until the MFMAs are done
  mfma_fence();
  pin_v(SA);
  pin_v(SB);
  pin_v(dPA);
  pin_v(dPB);
  wait_vmem<0>();   // no copy may still be writing this workgroup's LDS when it ends
  // dV/dK of the last step (its rows are in slot (nsteps-1) % NR)
  {
    const bool odd_last = (nsteps - 1) & 1;
    const uint32_t Ql = (uint32_t)((nsteps - 1) % NR) * 2 * QB, dOl = Ql + QB;   // slot of step nsteps-1
    auto last = [&](const bf16x8 (&Pl)[2], const bf16x8 (&Sl)[2]) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < NT; ++u) {   // the first PF fragments were read by the last iteration
        const int t2 = u / DB, nb = u % DB;
        const bf16x8 tv = u < PF ? ftv[u] : ld_t(dOl, u), tk = u < PF ? ftk[u] : ld_t(Ql, u);
        mma_a(dv[nb], Pl[t2], tv);
        mma_a(dk[nb], Sl[t2], tk);
      }
    };
    // one code path: the last step's P and dS (packed, and in fp32 for the remainders) are moved
    // into the even buffers first
    if (odd_last) {
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) {
        PA[t2] = PB[t2];
        DSA[t2] = DSB[t2];
      }
      if constexpr (REM) {
        SA = SB;
        dPA = dPB;
      }
    }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      anchor(PA[t2]);
      anchor(DSA[t2]);
    }
    valu_fence();
    last(PA, DSA);
    if constexpr (REM) remainders(SA, dPA, PA, DSA, Ql, dOl);
    mfma_fence();
#pragma unroll
    for (int nb = 0; nb < DB; ++nb) {
      pin_a(dk[nb]);
      pin_a(dv[nb]);
    }
  }

  // accumulator layout: lane <-> head_dim column 32*nb + l32, element v <-> key of the wave
  const float scale = a.s.scale;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int key = 32 * wave + 8 * (v >> 2) + 4 * hh + (v & 3);
    if (key >= it.nk) continue;
    float* kdst;
    float* vdst;
    if (it.part < 0) {
      const size_t o = (size_t)a.plan.kv_list[it.kv_off + key] * a.s.hkv * D + (size_t)hk * D;
      kdst = a.dK + o;
      vdst = a.dV + o;
    } else {
      const size_t o = ((size_t)it.part * BKV_TILE + key) * D;
      kdst = a.part_dk + o;
      vdst = a.part_dv + o;
    }
    if (it.part < 0 && it.acc) {   // a cached node's keys: add to the gradients of earlier calls
#pragma unroll
      for (int nb = 0; nb < DB; ++nb) {
        kdst[32 * nb + l32] += dk[nb][v] * scale;
        vdst[32 * nb + l32] += dv[nb][v];
      }
    } else {
#pragma unroll
      for (int nb = 0; nb < DB; ++nb) {
        kdst[32 * nb + l32] = dk[nb][v] * scale;
        vdst[32 * nb + l32] = dv[nb][v];
      }
    }
  }
}

// ============================================================================================
// bf16 dQ kernel (the structure of the forward kernel).  A wavefront holds Q, dO and the dQ
// accumulators of NH 32-row halves of one head in AGPRs and the scores in VGPRs; with NH = 2,
// one wavefront per SIMD, and every K or V fragment read from LDS feeds two MFMAs.  Stage j
// issues the S = K Q^T and dP = V dO^T MFMAs of 32-key block j+1 and the dQ^T += K^T dS^T MFMAs
// of block j-1, and between them computes P = exp2(S c - LSE log2 e) and dS = P (dP - Delta) of
// block j.
template <int D, int NW, int NS, int NH>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(3 - NH, 3 - NH))) void bwd_dq_bf16_w64_kernel(BwdArgs a) {
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;
  constexpr int RPI = 64 / CPR;
  constexpr int TB = KV_TILE * RB;
  constexpr int NI = KV_TILE / RPI;
  constexpr int IPW = NI / NW;
  constexpr int KS = D / 16;                     // S (and dP) MFMAs per row half and block
  constexpr int DB = D / 32;
  constexpr int NDQ = 2 * DB;                    // dQ MFMAs per row half and block
  constexpr int TPB = IDX_BLK / KV_TILE;
  constexpr int CPW = 2 * IPW;
  static_assert(NI % NW == 0 && (NS == 3 || NS == 4) && NS - 1 <= TPB, "tile copy split / ring depth");
  static_assert(D == 128 || D == 64, "head_dim");
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
  float lse2[NH], del[NH];
  // sum over this lane's keys of dS' = P (dP - Delta), with Delta = dO . O from the bf16 O: the
  // row's total is Delta' - Delta, so that the dK/dV pass can use the exact Delta' = sum_j P dP
  float eps[NH];
  bf16x8 qreg[NH][KS], doreg[NH][KS];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    ridx[rh] = (wave % rwn) * (32 * NH) + 32 * rh + l32;
    row_ok[rh] = ridx[rh] < it.nq;
    row[rh] = a.plan.q_list[it.q_off + (row_ok[rh] ? ridx[rh] : it.nq - 1)];
    lim[rh] = min(nkv - 1, a.plan.row_pos[row[rh]] - it.kv_pos0);
    lse2[rh] = a.lse2[(size_t)row[rh] * a.s.hq + head];
    del[rh] = a.delta[(size_t)row[rh] * a.s.hq + head];
    const size_t o = ((size_t)row[rh] * a.s.hq + head) * D + 8 * hh;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      qreg[rh][s] = as_bf(ld16((const bf16_t*)a.Q + o + 16 * s));
      doreg[rh][s] = as_bf(ld16((const bf16_t*)a.dO + o + 16 * s));
    }
  }

  // dP accumulators start at -Delta: one MFMA of A = 1 on k = 0, 1 (every key) and B = the (hi, lo)
  // bf16 split of the column's -Delta on k = 0, 1 (zero on lanes 32-63, which hold k = 8..15)
  const bf16x8 ones_k01 = as_bf(hh ? u32x4{0u, 0u, 0u, 0u} : u32x4{0x3F803F80u, 0u, 0u, 0u});
  bf16x8 ndel[NH];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    ndel[rh] = as_bf(u32x4{hh ? 0u : split_bf16(-del[rh]), 0u, 0u, 0u});
    eps[rh] = 0.f;
  }
  // LDS byte offsets of this lane's fragments inside a 32-key block (gtile_off layout): K or V
  // fragment s (rows l32, chunk 2s + hh) at koff[s & 1] + 1024 (s >> 1); K^T fragment of k-step
  // t2 and d block mb (rows 16 t2 + 8 rd + 4 hh + r4, chunks 4 mb + (dsub + 4 j) / 8) at
  // toff[rd] + 16 t2 RB + 1024 mb
  const int koff[2] = {gtile_off<D>(l32, hh), gtile_off<D>(l32, 2 + hh)};
  int toff[2];
  {
    const int r4 = (lane & 15) >> 2, j = lane & 3, dsub = 16 * ((lane >> 4) & 1);
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) toff[rd] = gtile_off<D>(8 * rd + 4 * hh + r4, (dsub + 4 * j) >> 3) + 8 * (j & 1);
  }
  static_assert(NW * NH == 8 && IPW * NW == CPR, "copies: NW / 4 waves per row group of a tile, IPW units each");

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
  // all copies into ring slot t % NS, of tile min(t, ntiles - 1) (see the forward kernel)
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

  f32x16 dq[NH][DB];
#pragma unroll
  for (int rh = 0; rh < NH; ++rh)
#pragma unroll
    for (int mb = 0; mb < DB; ++mb) {
      dq[rh][mb] = f32x16{};
      pin_a(dq[rh][mb]);
    }
#pragma unroll
  for (int rh = 0; rh < NH; ++rh)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      pin_a(qreg[rh][s]);
      pin_a(doreg[rh][s]);
    }
  valu_fence();
  const float c = a.s.scale * kLog2e;

  auto mask_elem = [&](f32x16 (&S)[NH], int rh, int v, int kb) __attribute__((always_inline)) {
    const int x = lim[rh] - kb - 4 * hh;    // element v holds key kb + 4*hh + 8*(v/4) + v%4
    S[rh][v] = (8 * (v >> 2) + (v & 3) > x) ? kNegInf : S[rh][v];
  };
  // ---- one stage.  Sc, dPc: block j (dS now); Sn, dPn: block j+1 (MFMAs now, K and V rows at
  // Kn, Vn); dSp: dS of block j-1 (dQ MFMAs now, K rows at Kp); dSc: block j's dS (written).
  auto stage = [&](f32x16 (&Sc)[NH], f32x16 (&dPc)[NH], f32x16 (&Sn)[NH], f32x16 (&dPn)[NH],
                   const bf16x8 (&dSp)[NH][2], bf16x8 (&dSc)[NH][2], const uint8_t* Kn, const uint8_t* Vn,
                   const uint8_t* Kp, int kb, auto masked, auto extra, auto dq_first) __attribute__((always_inline)) {
    // element e = 16 rh + v: scaled and shifted at chunk F(e), exponentiated at F(e)+1,
    // multiplied by dP - Delta at F(e)+2; each 8-element group is packed after its last product
    auto F = [](int e) constexpr { return (e * 29) / (16 * NH); };
    auto chunk = [&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      static_for<16 * NH>([&](auto ec) __attribute__((always_inline)) {
        constexpr int e = decltype(ec)::value, rh = e / 16, v = e % 16;
        if constexpr (F(e) == q) {
          if constexpr (decltype(masked)::value) mask_elem(Sc, rh, v, kb);
          Sc[rh][v] = fmaf(Sc[rh][v], c, -lse2[rh]);
        }
        if constexpr (F(e) + 1 == q) Sc[rh][v] = fast_exp2(Sc[rh][v]);
        if constexpr (F(e) + 2 == q) {
          dPc[rh][v] = Sc[rh][v] * dPc[rh][v];
          eps[rh] += dPc[rh][v];
          anchor(eps[rh]);   // (else the compiler gathers the 32 dependent adds in one block)
        }
        if constexpr (v % 8 == 7 && F(e) + 2 == q) {
          dSc[rh][v / 8] = pack8(dPc[rh], 8 * (v / 8));
          anchor(dSc[rh][v / 8]);
        }
      });
    };
    static_assert(F(16 * NH - 1) + 2 <= 31, "dS schedule");
    bf16x8 kf[KS], vf[KS], tf[NDQ];
    auto load_k = [&](int s) __attribute__((always_inline)) {
      kf[s] = as_bf(ld16(Kn + koff[s & 1] + (s >> 1) * 1024));
      vf[s] = as_bf(ld16(Vn + koff[s & 1] + (s >> 1) * 1024));
    };
    auto load_t = [&](int u) __attribute__((always_inline)) {   // u = DB * t2 + mb
      const int t2 = u / DB, mb = u % DB;
      const int o = 16 * t2 * RB + 1024 * mb;
      tf[u] = as_bf(lds_tr(Kp + toff[0] + o), lds_tr(Kp + toff[1] + o));
    };
    // fragments in use order: (K, V) pairs of the S and dP MFMAs and K^T fragments of the dQ
    // MFMAs, in the order the stage issues them; each is read PF pairs ahead
    constexpr bool DQF = decltype(dq_first)::value;
    constexpr int PF = PSATTN_DQ_PF;
    auto load_frag = [&](int f) __attribute__((always_inline)) {
      if (DQF) {
        if (f < NDQ) load_t(f);
        else if (f < NDQ + KS) load_k(f - NDQ);
      } else {
        if (f < KS) load_k(f);
        else if (f < KS + NDQ) load_t(f - KS);
      }
    };
#pragma unroll
    for (int f = 0; f < PF; ++f) load_frag(f);
    constexpr int NS_SLOTS = NH + 2 * NH * KS, NQ_SLOTS = NH * NDQ, NSLOT = NS_SLOTS + NQ_SLOTS;
    auto slot = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      constexpr int is = DQF ? (i >= NQ_SLOTS ? i - NQ_SLOTS : -1) : (i < NS_SLOTS ? i : -1);   // S/dP slot
      constexpr int iq = DQF ? (i < NQ_SLOTS ? i : -1) : (i >= NS_SLOTS ? i - NS_SLOTS : -1);   // dQ slot
      if constexpr (is >= 0 && is < NH) {
        mma_vv_first(dPn[is], ones_k01, ndel[is]);   // dP starts at -Delta
      } else if constexpr (is >= 0) {
        constexpr int s = (is - NH) / (2 * NH), w = (is - NH) % (2 * NH), rh = w % NH;   // w < NH: S, else dP
        if constexpr (w == 0) load_frag((DQF ? NDQ : 0) + s + PF);
        if constexpr (w < NH) {
          if constexpr (s == 0) mma_v_first(Sn[rh], kf[s], qreg[rh][s]);
          else mma_v(Sn[rh], kf[s], qreg[rh][s]);
        } else {
          mma_v(dPn[rh], vf[s], doreg[rh][s]);
        }
      } else {
        constexpr int u = iq / NH, rh = iq % NH;
        constexpr int t2 = u / DB, mb = u % DB;
        if constexpr (rh == 0) load_frag((DQF ? 0 : KS) + u + PF);
        mma_a(dq[rh][mb], tf[u], dSp[rh][t2]);
      }
      static_for<(32 * (i + 1)) / NSLOT - (32 * i) / NSLOT>([&](auto dq_) __attribute__((always_inline)) {
        chunk(IntC<(32 * i) / NSLOT + decltype(dq_)::value>{});
      });
      extra(ic);
      sched_fence();
    };
    static_for<NSLOT>(slot);
  };

  wait_vmem<0>();
  __syncthreads();
#pragma unroll
  for (int p = 0; p < NS - 1; ++p) issue(p);
  wait_vmem<CPW * (NS - 2)>();
  __syncthreads();

  f32x16 SA[NH], SB[NH], dPA[NH], dPB[NH];
  bf16x8 dSA[NH][2], dSB[NH][2];
  // block 0's S and dP; block -1's dS is zero (its dQ products, on tile 0's K rows, add nothing)
  {
    const uint8_t* K0 = &smem[0][0][0];
    const uint8_t* V0 = &smem[0][1][0];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8 k = as_bf(ld16(K0 + koff[s & 1] + (s >> 1) * 1024));
      const bf16x8 v = as_bf(ld16(V0 + koff[s & 1] + (s >> 1) * 1024));
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) {
        if (s == 0) {
          mma_v_first(SA[rh], k, qreg[rh][s]);
          mma_vv_first(dPA[rh], ones_k01, ndel[rh]);
          mma_v(dPA[rh], v, doreg[rh][s]);
        } else {
          mma_v(SA[rh], k, qreg[rh][s]);
          mma_v(dPA[rh], v, doreg[rh][s]);
        }
      }
    }
#pragma unroll
    for (int rh = 0; rh < NH; ++rh)
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2) dSB[rh][t2] = bf16x8{};
    mfma_fence();
  }

  // Tile t+NS-1 is copied during tile t: its V rows in stage 2t (V of tile t-1 was last read by
  // the dP products of block 2t-1, before the previous barrier), its K rows in stage 2t+1
  // (after the barrier that ends the dQ products of block 2t-1 on K of tile t-1).
  auto tile = [&](int t, auto masked) __attribute__((always_inline)) {
    const uint8_t* Kt = &smem[t % NS][0][0];
    const uint8_t* Vt = &smem[t % NS][1][0];
    const uint8_t* Kprev = t > 0 ? &smem[(t + NS - 1) % NS][0][0] + 32 * RB : Kt;
    const int tn = t + NS - 1;
    const int slot = issue_slot(min(tn, ntiles - 1));
    auto vcopies = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i % 6 == 3 && i / 6 < IPW) issue_copy1(tn % NS, IntC<i / 6>{}, slot, 1);
    };
    // stage 2t: S, dP of block 2t+1, dQ of block 2t-1, dS of block 2t; V copies
    stage(SA, dPA, SB, dPB, dSB, dSA, Kt + 32 * RB, Vt + 32 * RB, Kprev, t * KV_TILE, masked, vcopies, Flag<false>{});
    wait_vmem<(2 * NS - 5) * IPW>();
    __syncthreads();
    auto kcopies = [&](auto ic) __attribute__((always_inline)) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i % 6 == 3 && i / 6 < IPW) issue_copy1(tn % NS, IntC<i / 6>{}, slot, 0);
      if constexpr (i == 6 * IPW + 3) {
        if (tn < ntiles && tn % TPB == 0 && tn >= TPB) fetch_index_block(tn / TPB + 1);
      }
    };
    // stage 2t+1: dQ of block 2t first (K rows resident before the barrier), then S, dP of block
    // 2t+2 (tile t+1; unused past the last tile), dS of block 2t+1; K copies
    stage(SB, dPB, SA, dPA, dSA, dSB, &smem[(t + 1) % NS][0][0], &smem[(t + 1) % NS][1][0], Kt,
          t * KV_TILE + 32, masked, kcopies, Flag<true>{});
  };
  int t = 0;
  for (; t < min(it.nfull, ntiles); ++t) tile(t, Flag<false>{});
  for (; t < ntiles; ++t) tile(t, Flag<true>{});
  // the last stage's S and dP MFMAs (of the block past the end) have no readers: their registers
  // may be reused at once, so let them finish first (scheduling barriers keep the epilogue's
  // address arithmetic behind the wait states)
  sched_fence();
  mfma_fence();
  sched_fence();
  wait_vmem<0>();   // no copy may still be writing this workgroup's LDS when it ends
  // dQ of the last block
  {
    const uint8_t* Kl = &smem[(ntiles - 1) % NS][0][0] + 32 * RB;
#pragma unroll
    for (int u = 0; u < NDQ; ++u) {
      const int t2 = u / DB, mb = u % DB;
      const int o = 16 * t2 * RB + 1024 * mb;
      const bf16x8 k = as_bf(lds_tr(Kl + toff[0] + o), lds_tr(Kl + toff[1] + o));
#pragma unroll
      for (int rh = 0; rh < NH; ++rh) mma_a(dq[rh][mb], k, dSB[rh][t2]);
    }
    mfma_fence();
#pragma unroll
    for (int rh = 0; rh < NH; ++rh)
#pragma unroll
      for (int mb = 0; mb < DB; ++mb) pin_a(dq[rh][mb]);
  }
  // the exact Delta' = Delta + (row sum of dS'), as the (hi, lo) bf16 start value -Delta' of the
  // dK/dV kernel's dP accumulators; a row whose key range was split leaves its part of the sum to
  // the fixed-order reduction of the pieces
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    const float e = pair_sum(eps[rh]);   // lanes l and l ^ 32 hold different keys of one row
    if (hh == 0 && row_ok[rh]) {
      if (it.part < 0) {
        const uint32_t w = split_bf16(-del[rh]);
        const float d0 = bf2f(w & 0xffffu) + bf2f(w >> 16);   // the -Delta the dP products started from
        ((uint32_t*)a.kv_nd)[(size_t)row[rh] * a.s.hq + head] = split_bf16(d0 - e);
      } else {
        a.part_eps[((size_t)it.part + ridx[rh]) * a.s.hq + head] = e;
      }
    }
  }

  // dQ rows leave as whole fp32 rows: each wave stages one 32-row half at a time in its own part of
  // the LDS ring (free once every wave has finished the dQ products above; padded row stride QS),
  // then copies it out 16 bytes per lane, two rows per instruction.  The destination of staged
  // row r comes from lane r of the half.
  // (Forms whose staged halves would not fit the ring store straight from the accumulators.)
  constexpr int QS = D * 4 + 16;
  constexpr int CPRQ = D * 4 / 16, RPIQ = 64 / CPRQ;   // 16-byte chunks per row, rows per instruction
  const float scale = a.s.scale;
  if constexpr (NW * 32 * QS > NS * 2 * TB) {
#pragma unroll
    for (int rh = 0; rh < NH; ++rh) {
      if (!row_ok[rh]) continue;
      float* dst = it.part < 0 ? a.dQ + ((size_t)row[rh] * a.s.hq + head) * D
                               : a.part_dq + (((size_t)it.part + ridx[rh]) * a.s.hq + head) * D;
#pragma unroll
      for (int mb = 0; mb < DB; ++mb)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          *(f32x4*)(dst + 32 * mb + 8 * g4 + 4 * hh) =
              f32x4{dq[rh][mb][4 * g4] * scale, dq[rh][mb][4 * g4 + 1] * scale, dq[rh][mb][4 * g4 + 2] * scale,
                    dq[rh][mb][4 * g4 + 3] * scale};
    }
    return;
  }
  uint8_t* qt = &smem[0][0][0] + wave * 32 * QS;
  __syncthreads();
#pragma unroll
  for (int rh = 0; rh < NH; ++rh) {
    uint8_t* qrow = qt + l32 * QS;
#pragma unroll
    for (int mb = 0; mb < DB; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4)
        *(f32x4*)(qrow + 4 * (32 * mb + 8 * g4 + 4 * hh)) =
            f32x4{dq[rh][mb][4 * g4] * scale, dq[rh][mb][4 * g4 + 1] * scale, dq[rh][mb][4 * g4 + 2] * scale,
                  dq[rh][mb][4 * g4 + 3] * scale};
    const size_t dsto = it.part < 0 ? ((size_t)row[rh] * a.s.hq + head) * D
                                    : (((size_t)it.part + ridx[rh]) * a.s.hq + head) * D;
    float* const base = it.part < 0 ? a.dQ : a.part_dq;
    const int ch = lane % CPRQ;
#pragma unroll
    for (int k = 0; k < 32 / RPIQ; ++k) {
      const int rl = k * RPIQ + lane / CPRQ;
      const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)dsto, rl);
      const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(dsto >> 32), rl);
      const int ok = __shfl((int)row_ok[rh], rl);
      const u32x4 v = *(const u32x4*)(qt + rl * QS + 16 * ch);
      if (ok) *(u32x4*)(base + (((size_t)hi << 32) | lo) + 4 * ch) = v;
    }
  }
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
        s_del[tid] = a.delta[(size_t)row * a.s.hq + head];
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
  const bool acc = it.part < 0 && it.acc;   // a cached node's keys: add to earlier calls' gradients
#pragma unroll
  for (int i = 0; i < H; ++i) {
    kd[i] = dk[i] * a.s.scale + (acc ? kd[i] : 0.f);
    vd[i] = dv[i] + (acc ? vd[i] : 0.f);
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
  const float del = a.delta[(size_t)row * a.s.hq + head];
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
// Delta = rowsum(dO * O) per (row, head) (O + O_lo when the forward's residual is given),
// LSE * log2(e) for the exp2-based kernels, and the (hi, lo) start values of the dK/dV kernel's
// accumulators.  (row, head) pairs are walked in memory order (O, dO and O_lo are [Ns][Hq][d], the
// statistics [Ns][Hq]): D/8 lanes per pair, 8 elements each, so that every pass of a workgroup
// reads one contiguous span of each tensor and writes one run of each statistic; every lane issues
// all its loads before the first product.  One pass per workgroup measured fastest (against two
// and four: more workgroups in flight hide more of the load latency than more loads per lane).
constexpr int PRE_PASSES = 1;
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_pre_kernel(BwdArgs a) {
  const int D = a.s.d, hq = a.s.hq, ns = a.s.ns;
  const int lanes = D / 8;
  const int per_pass = 256 / lanes;
  const int64_t npairs = (int64_t)ns * hq;
  const int64_t pair0 = (int64_t)blockIdx.x * per_pass * PRE_PASSES + threadIdx.x / lanes;
  const int sub = threadIdx.x % lanes;
  float acc[PRE_PASSES];
  if (BF16) {
    // O + O_lo (two bf16 whose fp32 sum is exact) when the forward's rounding residual is given
    u32x4 x[PRE_PASSES], y[PRE_PASSES], z[PRE_PASSES];
    const bool res = a.O_lo != nullptr;
#pragma unroll
    for (int p = 0; p < PRE_PASSES; ++p) {
      const size_t o = (size_t)min(pair0 + p * per_pass, npairs - 1) * D + sub * 8;
      x[p] = ld16((const bf16_t*)a.O + o);
      y[p] = ld16((const bf16_t*)a.dO + o);
      z[p] = res ? ld16((const bf16_t*)a.O_lo + o) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int p = 0; p < PRE_PASSES; ++p) {
      acc[p] = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[p] = fmaf(bf2f(x[p][e] & 0xffffu) + bf2f(z[p][e] & 0xffffu), bf2f(y[p][e] & 0xffffu), acc[p]);
        acc[p] = fmaf(bf2f(x[p][e] >> 16) + bf2f(z[p][e] >> 16), bf2f(y[p][e] >> 16), acc[p]);
      }
    }
  } else {
    f32x4 x[PRE_PASSES][2], y[PRE_PASSES][2];
#pragma unroll
    for (int p = 0; p < PRE_PASSES; ++p) {
      const size_t o = (size_t)min(pair0 + p * per_pass, npairs - 1) * D + sub * 8;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        x[p][k] = *(const f32x4*)((const float*)a.O + o + 4 * k);
        y[p][k] = *(const f32x4*)((const float*)a.dO + o + 4 * k);
      }
    }
#pragma unroll
    for (int p = 0; p < PRE_PASSES; ++p) {
      acc[p] = 0.f;
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[p] = fmaf(x[p][k][e], y[p][k][e], acc[p]);
    }
  }
#pragma unroll
  for (int p = 0; p < PRE_PASSES; ++p) {
    for (int w = lanes / 2; w >= 1; w >>= 1) acc[p] += __shfl_xor(acc[p], w);
    const int64_t pr = pair0 + p * per_pass;
    if (pr < npairs && sub == 0) {
      const int row = (int)(pr / hq), h = (int)(pr % hq);
      const float lse = a.LSE[(size_t)h * ns + row];
      a.delta[pr] = acc[p];   // the statistics are [Ns][Hq]: pair pr's entry, written in order
      a.lse2[pr] = lse * kLog2e;
      ((uint32_t*)a.kv_nls)[pr] = split_bf16(-lse / a.s.scale);
      ((uint32_t*)a.kv_nd)[pr] = split_bf16(-acc[p]);
    }
  }
}

// dK/dV = sum of partial tiles in ascending chunk order (added to dK/dV for a cached node's keys)
__global__ __launch_bounds__(256) void bwd_reduce_kv_kernel(BwdArgs a) {
  const ReduceEntry e = a.plan.reduce[blockIdx.x];
  const int D = a.s.d;
  const size_t kv_stride = (size_t)a.s.hkv * D;
  for (int idx = blockIdx.y * blockDim.x + threadIdx.x; idx < e.nk * (D / 4); idx += gridDim.y * blockDim.x) {
    const int k = idx / (D / 4), d4 = (idx % (D / 4)) * 4;
    f32x4 sk = f32x4{}, sv = f32x4{};
    for (int j = 0; j < e.nparts; ++j) {
      const size_t o = (((size_t)e.part0 + j) * BKV_TILE + k) * D + d4;
      sk += *(const f32x4*)(a.part_dk + o);
      sv += *(const f32x4*)(a.part_dv + o);
    }
    const size_t o = (size_t)a.plan.kv_list[e.kv_off + k] * kv_stride + (size_t)e.hk * D + d4;
    if (e.acc) {
      sk = *(const f32x4*)(a.dK + o) + sk;
      sv = *(const f32x4*)(a.dV + o) + sv;
    }
    *(f32x4*)(a.dK + o) = sk;
    *(f32x4*)(a.dV + o) = sv;
  }
}

// dQ = sum of partial rows in ascending piece order (bf16: also the pieces' row sums of dS', which
// complete the exact Delta' of the dK/dV kernel, as the dQ kernel does for unsplit rows)
template <bool BF16>
__global__ __launch_bounds__(256) void bwd_reduce_dq_kernel(BwdArgs a) {
  const MergeEntry e = a.plan.merge[blockIdx.x];
  const int D = a.s.d, hq = a.s.hq, bmq = a.s.bmq;
  const int per_row = hq * D / 4;
  if (BF16) {
    for (int idx = blockIdx.y * blockDim.x + threadIdx.x; idx < e.nq * hq; idx += gridDim.y * blockDim.x) {
      const int i = idx / hq, h = idx % hq;
      float s = 0.f;
      for (int j = 0; j < e.nparts; ++j) s += a.part_eps[((size_t)e.part0 + (size_t)j * bmq + i) * hq + h];
      uint32_t* nd = (uint32_t*)a.kv_nd + (size_t)a.plan.q_list[e.q_off + i] * hq + h;
      const uint32_t w = *nd;
      *nd = split_bf16(bf2f(w & 0xffffu) + bf2f(w >> 16) - s);
    }
  }
  for (int idx = blockIdx.y * blockDim.x + threadIdx.x; idx < e.nq * per_row; idx += gridDim.y * blockDim.x) {
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

hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16, hipStream_t st) {
  const int pairs_per_block = 256 / (a.s.d / 8) * PRE_PASSES;
  const dim3 grid((unsigned)(((int64_t)a.s.ns * a.s.hq + pairs_per_block - 1) / pairs_per_block));
  if (bf16) hipLaunchKernelGGL((bwd_pre_kernel<true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((bwd_pre_kernel<false>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_kv(const BwdArgs& a, bool bf16, hipStream_t st) {
  // (the bf16 kernel addresses the pools and the Q / dO tensors by 32-bit byte offsets; the host
  // rejects larger trees with PSATTN_E_UNSUPPORTED)
  const dim3 grid(a.n_bkv), block(256);
  if (bf16) {
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_kv_bf16_1w_kernel<128, PSATTN_KV_REM>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_kv_bf16_1w_kernel<64, PSATTN_KV_REM>), grid, block, 0, st, a);
  } else {
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_kv_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_kv_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq(const BwdArgs& a, bool bf16, hipStream_t st) {
  const dim3 grid(a.n_fwd);
  if (bf16) {
    // 8 / NH waves of NH*32 rows (the planner makes every item 8 (subtile, head) pairs)
    if (a.s.rw % PSATTN_DQ_NH != 0 || a.s.nw != 8) return hipErrorInvalidValue;
    constexpr int NW = 8 / PSATTN_DQ_NH;
    const dim3 block(NW * 64);
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_dq_bf16_w64_kernel<128, NW, 4, PSATTN_DQ_NH>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_dq_bf16_w64_kernel<64, NW, 4, PSATTN_DQ_NH>), grid, block, 0, st, a);
  } else {
    const dim3 block(2 * a.s.bmq * a.s.hc);
    if (a.s.d == 128) hipLaunchKernelGGL((bwd_dq_f32_kernel<128>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((bwd_dq_f32_kernel<64>), grid, block, 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_reduce_kv(const BwdArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(bwd_reduce_kv_kernel, dim3(a.n_reduce, kMergeSlices), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_reduce_dq(const BwdArgs& a, bool bf16, hipStream_t st) {
  if (bf16) hipLaunchKernelGGL(bwd_reduce_dq_kernel<true>, dim3(a.n_merge, kMergeSlices), dim3(256), 0, st, a);
  else hipLaunchKernelGGL(bwd_reduce_dq_kernel<false>, dim3(a.n_merge, kMergeSlices), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_bwd_zero_pad(const BwdArgs& a, hipStream_t st) {
  const int64_t n = (int64_t)a.n_pad * a.s.hkv * a.s.d / 4;
  const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(bwd_zero_pad_kernel, dim3(blocks), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace psattn
