// Internal definitions shared by the gfx950 kernels of libcertkv.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "certkv.h"

namespace certkv {

// Per-launch table of up to kMaxSeq sequences, passed by value as a kernel
// argument so that no host-to-device copy is needed for ragged batches.
constexpr int kMaxSeq = 48;
constexpr int kMaxDevices = 64;  // devices whose properties are cached

// Compute units of device dev (queried once; 0 if the query fails).
inline int device_cus(int dev) {
  static std::atomic<int> cus[kMaxDevices];
  if (dev < 0 || dev >= kMaxDevices) return 0;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

struct SeqTab {
  int32_t count;             // sequences in this launch
  int32_t first;             // global index of the first one
  int64_t start[kMaxSeq];    // token offset in the packed token axis
  int32_t len[kMaxSeq];      // n_b
  int32_t n_keep[kMaxSeq];   // live slots per head (incl. the slot)
  int64_t b_real[kMaxSeq];   // H * n_keep - H
  int32_t b_min[kMaxSeq];    // max(1, floor(alpha * B_real / H))
};

// Geometry common to all kernels.
struct Geo {
  int32_t L, B, H, G, D, w;
  int64_t T;                 // total tokens
  float scale;               // softmax scale (natural-log units)
  int32_t causal;
  int32_t keep_w;            // window keys ranked first (w), or 0
  int32_t* status;           // optional: set to CERTKV_ENONFINITE on a non-finite value
  int32_t stat;              // curve statistic: 0 centered, 1 uncentered, 2 tail mass
  int32_t slot;              // slot rows per unit in the packed cache (1, or 0 without)
};

// Record a non-finite value in the caller's status word (racing stores all
// write the same value).
__device__ __forceinline__ void report_nonfinite(const Geo& g) {
  if (g.status) *g.status = CERTKV_ENONFINITE;
}

// Record a segment longer than a caller's row bound (same racing-store rule).
__device__ __forceinline__ void report_range(const Geo& g) {
  if (g.status) *g.status = CERTKV_ERANGE;
}

__device__ __forceinline__ int64_t unit_index(const Geo& g, int l, int b, int h) {
  return ((int64_t)l * g.B + b) * g.H + h;
}

// scores / curves / perm layout [L][H][T]: start of unit (l, b, h).
__device__ __forceinline__ int64_t lht_base(const Geo& g, int l, int h, int64_t tok0) {
  return ((int64_t)l * g.H + h) * g.T + tok0;
}

// Raw buffer resource over [base, base + bytes): loads through it take a
// uniform 64-bit base and a 32-bit per-lane byte offset, and return zero for
// offsets at or beyond `bytes` (hardware range check).
typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint32_t buf_load_u32(BufRsrc r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint32_t buf_load_u16(BufRsrc r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, 0);
}
__device__ __forceinline__ uint2 buf_load_u64(BufRsrc r, uint32_t off) {
  auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
  return make_uint2(v[0], v[1]);
}
__device__ __forceinline__ uint4 buf_load_u128(BufRsrc r, uint32_t off) {
  auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void buf_store_u32(BufRsrc r, uint32_t off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, 0);
}
// The same loads with a wave-uniform byte offset `soff` (held in the
// instruction's scalar offset; only `off` is range-checked, so the caller
// keeps soff + off inside the buffer).
__device__ __forceinline__ uint32_t buf_load_u32s(BufRsrc r, uint32_t off, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, (int)soff, 0);
}
__device__ __forceinline__ uint32_t buf_load_u16s(BufRsrc r, uint32_t off, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, (int)off, (int)soff, 0);
}
__device__ __forceinline__ uint2 buf_load_u64s(BufRsrc r, uint32_t off, uint32_t soff) {
  auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, (int)soff, 0);
  return make_uint2(v[0], v[1]);
}

// bf16 <-> fp32.  bf16 is the upper half of an IEEE binary32.
__device__ __forceinline__ float bf16_lo(uint32_t packed) { return __uint_as_float(packed << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t packed) { return __uint_as_float(packed & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }

// Round-to-nearest-even fp32 -> bf16 (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Descending-order radix key of a float: larger value -> smaller key, so an
// ascending stable sort of keys orders scores descending with ties kept in
// position order.  -0.0 takes the key of +0.0: the two compare equal, so
// they tie and keep position order like any other pair of equal scores.
__device__ __forceinline__ uint32_t desc_key(float f) {
  uint32_t u = __float_as_uint(f);
  u = (u << 1) ? u : 0u;
  uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ~asc;
}
__device__ __forceinline__ float desc_key_value(uint32_t key) {
  uint32_t asc = ~key;
  uint32_t u = (asc & 0x80000000u) ? (asc & 0x7fffffffu) : ~asc;
  return __uint_as_float(u);
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// fp64 shuffle across the wave (two 32-bit bpermutes).
__device__ __forceinline__ double shfl_xor_f64(double x, int mask) {
  return __shfl_xor(x, mask, 64);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

template <typename T>
__device__ __forceinline__ T wave_max(T x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    T y = __shfl_xor(x, m, 64);
    x = x > y ? x : y;
  }
  return x;
}

__device__ __forceinline__ float wave_min_f(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = fminf(x, __shfl_xor(x, m, 64));
  return x;
}

}  // namespace certkv

// Host-side launch helpers (defined in api.hip).
namespace certkv {
void prof_begin(const char* name, hipStream_t s);
void prof_end(hipStream_t s);
}  // namespace certkv

#define CERTKV_LAUNCH(name, kernel, grid, block, shmem, stream, ...)        \
  do {                                                                      \
    ::certkv::prof_begin(name, stream);                                     \
    hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);    \
    ::certkv::prof_end(stream);                                             \
    if (hipGetLastError() != hipSuccess) return CERTKV_EHIP;                \
  } while (0)
