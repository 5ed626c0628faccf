// Kernel launchers (defined in psattn_fwd.hip, psattn_bwd.hip and psattn_layer.hip, called by the C ABI).
#pragma once
#include <hip/hip_runtime.h>

#include "psattn_plan.h"

namespace psattn {

struct FwdArgs {
  PlanView plan;
  Shape s;
  int32_t n_items, n_merge;
  const void* Q;
  const void* K;
  const void* V;
  void* O;
  void* O_lo;       // bf16: residual O - bf16(O) of the fp32 result [Ns][Hq][d], or null
  float* LSE;
  float* part_o;    // [partial rows][Hq][d]
  float* part_lse;  // [partial rows][Hq]
  int64_t pool_slots;  // rows of the K and V pools
};

struct BwdArgs {
  PlanView plan;
  Shape s;
  int32_t n_fwd, n_merge, n_bkv, n_reduce, n_pad;
  const void* Q;
  const void* K;
  const void* V;
  const void* O;
  const void* O_lo; // bf16: residual of O (Delta from O + O_lo), or null
  const float* LSE;
  const void* dO;
  float* dQ;
  float* dK;
  float* dV;
  float* delta;    // [Ns][Hq]
  float* lse2;     // [Ns][Hq] LSE * log2(e)
  float* kv_nls;   // [Ns][Hq] -LSE / scale   (start of the dK/dV kernels' S accumulators)
  float* kv_nd;    // [Ns][Hq] -Delta         (start of their dP accumulators; bf16: the exact
                   //                          Delta' from the dQ pass, which runs first)
  float* part_dq;  // [partial rows][Hq][d]
  float* part_eps; // [partial rows][Hq] row sums of dS' of each piece (bf16)
  float* part_dk;  // [partial tiles][BKV_TILE][d]; each tile belongs to one kv head
  float* part_dv;
  int64_t pool_slots;  // rows of the K and V pools
};

// Each launcher enqueues one kernel on stream and returns the launch status.
hipError_t launch_fwd_main(const FwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_fwd_merge(const FwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_bwd_pre(const BwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_bwd_kv(const BwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_bwd_dq(const BwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_bwd_reduce_kv(const BwdArgs& a, hipStream_t st);
hipError_t launch_bwd_reduce_dq(const BwdArgs& a, bool bf16, hipStream_t st);
hipError_t launch_bwd_zero_pad(const BwdArgs& a, hipStream_t st);
// layer steps around the attention (psattn_layer.hip)
hipError_t launch_rope(const PlanView& plan, int32_t ns, int32_t heads, int32_t d, float theta, bool inverse, bool bf16,
                       void* X, hipStream_t st);
hipError_t launch_kv_move(const PlanView& plan, int32_t ns, int32_t row_bytes, bool to_pool, const void* a0,
                          const void* a1, void* b0, void* b1, hipStream_t st);

}  // namespace psattn
