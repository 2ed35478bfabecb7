// csr_device.h -- device helpers shared by the CSR SGD kernels: raw buffer
// views of one worker's arrays, the loss coefficient and step size, fp64
// row sums over 16 DPP lanes, and the per-lane row registers of a step.
#pragma once

#include <cmath>

#include "asap_launch.h"

namespace asap {
namespace csr {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kRowLanes = 16;                        // lanes per row on the fast path
constexpr int kFastRows = kWaves * 64 / kRowLanes;   // 64 rows per step

// Raw buffer resources over one worker's arrays: 32-bit byte offsets keep a
// lane's address in one register, and offsets past the end read 0.
constexpr int kRsrcWord3 = 0x00020000;  // gfx9-family raw buffer

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, int(bytes), kRsrcWord3);
}
__device__ __forceinline__ int ld_i32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ float ld_f32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void st_f32(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, off, 0, 0);
}

// Buffer views of one worker: nonzeros [seg, seg + nnz_w) and its model row.
struct Views {
  __amdgpu_buffer_rsrc_t code, val, model;
  long long seg;
};

__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// d loss(y m) / d m from an fp64 margin: the hinge decision y m < 1 is taken
// in fp64; the logistic factor 1 / (1 + e^{y m}) needs only fp32 accuracy.
__device__ __forceinline__ double loss_coef(double m, double y, int loss) {
  const double ym = y * m;
  if (loss == ASAP_LOSS_HINGE) return ym < 1.0 ? -y : 0.0;
  return -y / double(1.0f + expf(float(ym)));
}

__device__ __forceinline__ double step_size(int lr_kind, float lr0, int64_t t) {
  return lr_kind == 0 ? double(lr0) : double(lr0) / sqrt(double(t));
}

// Sum over the 16 lanes of a DPP row; every lane gets the same bits (each
// stage adds the same two operands in swapped order).
__device__ __forceinline__ double row16_sum(double v) {
#define ASAP_DPP_STAGE(ctrl)                                                                    \
  {                                                                                             \
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), ctrl, 0xF, 0xF, false);   \
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), ctrl, 0xF, 0xF, false);   \
    v += __hiloint2double(hi, lo);                                                              \
  }
  ASAP_DPP_STAGE(0xB1)   // quad_perm [1,0,3,2]
  ASAP_DPP_STAGE(0x4E)   // quad_perm [2,3,0,1]
  ASAP_DPP_STAGE(0x141)  // row_half_mirror
  ASAP_DPP_STAGE(0x140)  // row_mirror
#undef ASAP_DPP_STAGE
  return v;
}

__device__ __forceinline__ int row16_sum_i(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  return v;
}

__device__ __forceinline__ bool is_hot(int code) { return code <= -2; }
__device__ __forceinline__ int hot_slot(int code) { return -code - 2; }

// Raw nonzeros of one lane's share of one fast-path row (entries sub,
// sub+16, ...): ok bit j says entry j exists, kRowExists that the row does,
// kRowLong that it has more than 16*E nonzeros.
constexpr uint32_t kRowExists = 1u << 31;
constexpr uint32_t kRowLong = 1u << 30;

template <int E>
struct DataReg {
  int code[E];
  float val[E];
  uint32_t ok;
  float y;
};

__device__ __forceinline__ bool row_valid(const SgdArgs& a, int64_t k, int64_t K, int b) {
  return k < K && b < int(min(int64_t(a.batch), a.S - k * a.batch));
}

// Row descriptor of step k, fast-path row b, as loaded (row 0 when the row
// does not exist; nothing is computed on it until the next step).
__device__ __forceinline__ RowInfo load_row(const SgdArgs& a, const RowInfo* ri, int64_t k, int64_t K, int b) {
  return ri[row_valid(a, k, K, b) ? k * a.batch + b : 0];
}

template <int E>
__device__ __forceinline__ void load_data(const Views& w, const RowInfo& r, bool valid, int sub, DataReg<E>& d) {
  const int len = valid ? r.len : 0;
  const uint32_t st = uint32_t(r.start - w.seg);
  d.ok = (len > 0 ? kRowExists : 0u) | (len > kRowLanes * E ? kRowLong : 0u);
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const int e = sub + kRowLanes * j;
    const uint32_t p = e < len ? st + uint32_t(e) : 0u;
    d.code[j] = ld_i32(w.code, p * 4u);
    d.val[j] = ld_f32(w.val, p * 4u);
    d.ok |= uint32_t(e < len) << j;
  }
  d.y = r.y;
}

template <int E>
__device__ __forceinline__ int code_at(const DataReg<E>& d, int j) {
  return (d.ok >> j) & 1u ? d.code[j] : -1;
}

}  // namespace csr
}  // namespace asap
