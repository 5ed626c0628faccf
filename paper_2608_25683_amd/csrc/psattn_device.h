// Device-side helpers shared by the HIP kernels (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "psattn_launch.h"

namespace psattn {
namespace dev {

typedef uint16_t bf16_t;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) short s16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) float f32x2;

#define PSATTN_LDS(T, p) ((__attribute__((address_space(3))) T*)(p))

// compile-time flag passed to generic lambdas (if constexpr on decltype(flag)::value)
template <bool B>
struct Flag {
  static constexpr bool value = B;
};

// compile-time integer, and a loop that calls f(IntC<0>{}) .. f(IntC<N-1>{}) (fully unrolled)
template <int I>
struct IntC {
  static constexpr int value = I;
};
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IntC<I>{});
    static_for<N, I + 1>(f);
  }
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();
constexpr int IDX_BLK = 256;   // slot / row indices staged in LDS per block
constexpr int kMergeSlices = 8; // workgroups per merge / reduction record (grid y)
static_assert((IDX_BLK & (IDX_BLK - 1)) == 0, "staged index blocks are addressed modulo 2*IDX_BLK");

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ bf16x8 as_bf(const u32x4& v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ bf16x8 as_bf(const u32x2& lo, const u32x2& hi) {
  return __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
}
__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }
__device__ __forceinline__ u32x2 ld8(const void* p) { return *(const u32x2*)p; }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
// two floats -> two bf16 (round to nearest even) in one dword: a single v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}
__device__ __forceinline__ float bf2f(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
// x as hi + lo, two bf16 (hi the nearest bf16 to x, lo the nearest to x - hi), hi in the low half
__device__ __forceinline__ uint32_t split_bf16(float x) {
  const float hi = bf2f(pack2(x, 0.f) & 0xffffu);
  return pack2(x, x - hi);
}
// 8 consecutive accumulator values -> one bf16x8 MFMA operand
__device__ __forceinline__ bf16x8 pack8(const f32x16& x, int base) {
  u32x4 w;
  w[0] = pack2(x[base + 0], x[base + 1]);
  w[1] = pack2(x[base + 2], x[base + 3]);
  w[2] = pack2(x[base + 4], x[base + 5]);
  w[3] = pack2(x[base + 6], x[base + 7]);
  return as_bf(w);
}

// The remainders x - hi of the same 8 values, given hi = pack8(x, base): one bf16x8 operand that,
// added to hi in a product, carries x to ~2^-17 relative (hi's element 2k sits in the low half of
// dword k, element 2k+1 in the high half)
__device__ __forceinline__ bf16x8 pack8_rem(const f32x16& x, int base, const bf16x8& hi) {
  const u32x4 h = __builtin_bit_cast(u32x4, hi);
  u32x4 w;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    w[k] = pack2(x[base + 2 * k] - __uint_as_float(h[k] << 16), x[base + 2 * k + 1] - __uint_as_float(h[k] & 0xffff0000u));
  return as_bf(w);
}

// Max / sum over the lane pair (l, l ^ 32) with one v_permlane32_swap: whichever half the
// instruction exchanges, the two results hold this lane's value and its partner's.
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---- LDS tiles of rows of D bf16 (D*2 bytes per row), no padding.  The 16-byte chunk c of row
// r lives at chunk position c ^ swz(r), so that 16 consecutive rows read at one column, and
// 4 consecutive rows x 4 consecutive chunks read by the transposing loads, hit distinct banks.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (r >> 1) & 7;
}

// ---- LDS tiles of the one-wavefront-per-SIMD kernels (rows of D bf16).  Rows come in groups
// of 16.  A group is stored as 1 KB units, one per 4 consecutive 16-byte chunks: inside a unit
// the chunks follow each other (256 bytes apiece) and row r of chunk c sits at position
// (r mod 16) ^ 4 (c mod 4).  One copy instruction (64 lanes x 16 bytes) thus fills one unit with
// 64 bytes of each of 16 rows.  Reads of one chunk by 16 consecutive rows, and the transposing
// reads (4 rows x 4 chunks per 16 lanes, two such groups per 32 lanes), hit distinct banks, and
// the chunk offset of a fragment splits into a per-lane part and a multiple of 1 KB.
template <int D>
__device__ __forceinline__ int gtile_off(int r, int c) {
  return (r >> 4) * (16 * D * 2) + (c >> 2) * 1024 + (c & 3) * 256 + (((r & 15) ^ (4 * (c & 3))) << 4);
}

// 16 bytes per lane from global memory straight into LDS: lane i writes lds_base + 16 i.
// Issued through inline assembly so that the compiler does not wait for the copy before every
// later LDS read (it cannot tell which LDS bytes the copy writes); the kernels wait explicitly
// (wait_vmem + barrier) before reading a stage.  lds_base must be wave-uniform.
__device__ __forceinline__ void copy16_to_lds(const void* g, void* lds_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)PSATTN_LDS(void, lds_base));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
// As copy16_to_lds, with the LDS byte address given directly (wave-uniform).
__device__ __forceinline__ void copy16_to_lds_at(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
// As copy16_to_lds_at, reading 16 bytes at base + off for each lane (base wave-uniform, off a
// 32-bit byte offset per lane).
__device__ __forceinline__ void copy16_to_lds_off(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
// As copy16_to_lds_off, reading at base + off + OFF (OFF a compile-time byte offset), lane i
// still writing lds + 16 i.  The instruction offset is added to the LDS address as well as to the
// global one, so M0 is set to lds - OFF (lds >= OFF).
template <int OFF>
__device__ __forceinline__ void copy16_to_lds_off_imm(const void* base, uint32_t off, uint32_t lds) {
  static_assert(OFF >= 0 && OFF < 4096, "global instruction offset range");
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:%3" ::"v"(off), "s"(base), "s"(lds - OFF),
               "i"(OFF)
               : "memory", "m0");
}
// LDS byte address of a pointer into a __shared__ array (the low half of its generic address).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }
// 4 bytes per lane: lane i writes lds_base + 4 i (inactive lanes write nothing).
__device__ __forceinline__ void copy4_to_lds(const void* g, void* lds_base) {
  const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)PSATTN_LDS(void, lds_base));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
// copy4_to_lds with the LDS address given directly (wave-uniform)
__device__ __forceinline__ void copy4_to_lds_at(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds) : "memory", "m0");
}
// 4 bytes per lane from base + off (uniform base, 32-bit per-lane byte offset) to lds + 4 * lane
__device__ __forceinline__ void copy4_to_lds_off(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
// Wait until at most N vector-memory loads of this wave are in flight (gfx9 s_waitcnt encoding:
// vmcnt in bits 3:0 and 15:14, expcnt and lgkmcnt left at their maxima).  The intrinsic keeps
// the compiler's own load scoreboard in step, so it inserts no further waits for older loads.
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// Wait until at most N LDS (and scalar memory) operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_lds() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (N << 8));
}
// Workgroup barrier without the wait for this wave's outstanding LDS reads that __syncthreads
// adds; the memory clobber keeps the compiler from moving loads or stores across it.  LDS writes
// other waves must see after it need a wait_lds<0>() first.
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

// ---- MFMA through inline assembly, with the register class of each operand chosen here
// (accumulators and loop-invariant operands in AGPRs, scores in VGPRs).  The compiler does not
// treat these as matrix instructions, so the data hazards it would otherwise resolve are the
// caller's: a non-MFMA instruction may read or overwrite an MFMA result only 12 wait states after
// the MFMA that wrote it (see mfma_fence_a), and a register written by a VALU instruction may
// feed an MFMA only 2 wait states later.  Chained accumulation into the same registers needs
// no wait.
// d = a * b, d in VGPRs, b in AGPRs
__device__ __forceinline__ void mma_v_first(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(b));
}
// d += a * b, d in VGPRs, b in AGPRs
__device__ __forceinline__ void mma_v(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "a"(b));
}
// d = a * b, d, a and b in VGPRs
__device__ __forceinline__ void mma_vv_first(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "v"(b));
}
// d = a * b and d += a * b with d and b in AGPRs
__device__ __forceinline__ void mma_aa_first(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&a"(d) : "v"(a), "a"(b));
}
__device__ __forceinline__ void mma_aa(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(d) : "v"(a), "a"(b));
}
// d += a * b, d in AGPRs, a and b in VGPRs
__device__ __forceinline__ void mma_a(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(d) : "v"(a), "v"(b));
}
// Keep x in AGPRs from here on (an AGPR operand of the MFMAs above).
__device__ __forceinline__ void pin_a(bf16x8& x) { asm volatile("" : "+a"(x)); }
__device__ __forceinline__ void pin_a(f32x16& x) { asm volatile("" : "+a"(x)); }
// 12 wait states before later instructions may touch the results of the MFMAs issued so far;
// the accumulators passed to the following pin_a calls are then ordered after the wait.
__device__ __forceinline__ void mfma_fence() { asm volatile("s_nop 11"); }
// 2 wait states after VALU writes, before MFMAs read them.
__device__ __forceinline__ void valu_fence() { asm volatile("s_nop 1"); }
// Plain IEEE max without the quieting of signalling NaNs that fmaxf implies for operands the
// compiler cannot see the origin of (MFMA results from inline assembly).
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max3abs(float a, float b, float c) {   // max(a, |b|, |c|)
  float r;
  asm("v_max3_f32 %0, %1, |%2|, |%3|" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max2f(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// acc + lo + hi of a packed bf16 pair (one v_dot2c_f32_bf16 against (1, 1))
__device__ __forceinline__ float add_bf16_pair(uint32_t pair, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), one, acc, false);
}
// max over the lane pair (l, l ^ 32)
__device__ __forceinline__ float pair_max2(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max2f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Materialize x here: its computation cannot sink past this point.
__device__ __forceinline__ void anchor(float& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void anchor(f32x16& x) { asm volatile("" : "+v"(x)); }
// Move x to VGPRs here (from AGPRs, if it lives there).
__device__ __forceinline__ void pin_v(f32x16& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void anchor(bf16x8& x) { asm volatile("" : "+v"(x)); }
// Keep the scheduler from moving any instruction across this point.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Transposing LDS read: within each 16-lane group, lanes 4r..4r+3 point at 4 consecutive bf16 of
// row r (r = 0..3) and lane i of the group receives column i of those 4 rows.
__device__ __forceinline__ u32x2 lds_tr(const void* p) {
  s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(PSATTN_LDS(s16x4, p));
  return __builtin_bit_cast(u32x2, v);
}

}  // namespace dev
}  // namespace psattn
