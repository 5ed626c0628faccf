// The tree-dependent steps around the attention of one layer in the shared layout: rotary
// position embedding by each row's sequence position, K/V rows written into their pool slots
// (the page table), and dK/dV read back from the pool into row order.
//
// Rotary embedding: for sequence position p, the pair (x_i, x_{i + d/2}), i < d/2, turns by the
// angle p * theta^(-2i/d); the inverse (transposed) rotation, for the backward, turns by minus
// that angle.  Every token of a shared node has one position however many samples read it (the
// block's pos field, Sec. 6), so shared rows are rotated once.  Angles are formed and reduced in
// fp64 (positions reach 10^4 and beyond), the rotation itself is fp32.
#include <algorithm>

#include "psattn_device.h"

namespace psattn {
namespace {

using namespace dev;

template <bool BF16>
__global__ __launch_bounds__(256) void rope_kernel(PlanView plan, int32_t ns, int32_t heads, int32_t d, double log2_theta,
                                                   double sign, void* X) {
  const int half = d / 2;
  const int64_t n = (int64_t)ns * heads * half;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * blockDim.x) {
    const int i = (int)(idx % half);
    const int64_t rh = idx / half;
    const int row = (int)(rh / heads);
    const double ang = sign * (double)plan.row_pos[row] * exp2(-(2.0 * i / d) * log2_theta);
    double sd, cd;
    sincos(ang, &sd, &cd);
    const float s = (float)sd, c = (float)cd;
    const int64_t o0 = rh * d + i, o1 = o0 + half;
    if (BF16) {
      bf16_t* x = (bf16_t*)X;
      const float a = bf2f(x[o0]), b = bf2f(x[o1]);
      const uint32_t p = pack2(a * c - b * s, a * s + b * c);
      x[o0] = (bf16_t)(p & 0xffffu);
      x[o1] = (bf16_t)(p >> 16);
    } else {
      float* x = (float*)X;
      const float a = x[o0], b = x[o1];
      x[o0] = a * c - b * s;
      x[o1] = a * s + b * c;
    }
  }
}

// rows [Ns][hkv][d] <-> pool [slots][hkv][d], 16 bytes per thread
__global__ __launch_bounds__(256) void kv_move_kernel(PlanView plan, int32_t ns, int32_t row_bytes, int32_t to_pool,
                                                      const uint8_t* a0, const uint8_t* a1, uint8_t* b0, uint8_t* b1) {
  const int per_row = row_bytes / 16;
  const int64_t n = (int64_t)ns * per_row;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * blockDim.x) {
    const int row = (int)(idx / per_row), c = (int)(idx % per_row);
    const int64_t r_off = (int64_t)row * row_bytes + 16 * c;
    const int64_t p_off = (int64_t)plan.row_slot[row] * row_bytes + 16 * c;
    const int64_t src = to_pool ? r_off : p_off, dst = to_pool ? p_off : r_off;
    *(u32x4*)(b0 + dst) = *(const u32x4*)(a0 + src);
    *(u32x4*)(b1 + dst) = *(const u32x4*)(a1 + src);
  }
}

unsigned grid_for(int64_t n) { return (unsigned)std::min<int64_t>((n + 255) / 256, 8192); }

}  // namespace

hipError_t launch_rope(const PlanView& plan, int32_t ns, int32_t heads, int32_t d, float theta, bool inverse, bool bf16,
                       void* X, hipStream_t st) {
  const int64_t n = (int64_t)ns * heads * (d / 2);
  const double l2t = log2((double)theta), sign = inverse ? -1.0 : 1.0;
  if (bf16) hipLaunchKernelGGL(rope_kernel<true>, dim3(grid_for(n)), dim3(256), 0, st, plan, ns, heads, d, l2t, sign, X);
  else hipLaunchKernelGGL(rope_kernel<false>, dim3(grid_for(n)), dim3(256), 0, st, plan, ns, heads, d, l2t, sign, X);
  return hipGetLastError();
}

hipError_t launch_kv_move(const PlanView& plan, int32_t ns, int32_t row_bytes, bool to_pool, const void* a0,
                          const void* a1, void* b0, void* b1, hipStream_t st) {
  hipLaunchKernelGGL(kv_move_kernel, dim3(grid_for((int64_t)ns * (row_bytes / 16))), dim3(256), 0, st, plan, ns, row_bytes,
                     to_pool ? 1 : 0, (const uint8_t*)a0, (const uint8_t*)a1, (uint8_t*)b0, (uint8_t*)b1);
  return hipGetLastError();
}

}  // namespace psattn
