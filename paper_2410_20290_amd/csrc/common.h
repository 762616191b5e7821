// Shared device/host helpers of the Speculative Rejection library (gfx950).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdio>
#include <string>

typedef uint16_t bf16_t;  // bf16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace sr {

// ---- element conversions ---------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}
// Round to nearest even; NaN stays NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return 0x7FC0;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// Unpack 16 bytes into floats: 8 bf16 or 4 fp32.
template <typename T> struct Vec16;
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ __forceinline__ static void load(const bf16_t* p, float* out) {
    uint4 u = *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = __uint_as_float(w[i] << 16);
      out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ __forceinline__ static void load(const float* p, float* out) {
    float4 u = *reinterpret_cast<const float4*>(p);
    out[0] = u.x; out[1] = u.y; out[2] = u.z; out[3] = u.w;
  }
};

// One 16-byte-per-lane copy from memory straight into LDS
// (global_load_lds_dwordx4): lane l's 16 bytes land at lds_dst + 16 l bytes;
// lds_dst must be the same in every lane of the wave.  Counted by vmcnt.  A
// plain function, so that kernel templates can call it with dependent
// arguments.
__device__ __forceinline__ void dma16(const char* src, bf16_t* lds_dst) {
  __builtin_amdgcn_global_load_lds(src, lds_dst, 16, 0, 0);
}

// The same copy as a buffer load into LDS (buffer_load_dwordx4 ... lds): the
// source is base + voff + soff, with the base in a buffer resource (SGPRs),
// a 32-bit per-lane offset and a wave-uniform scalar offset, so no 64-bit
// address arithmetic per copy.  The resource is raw (no stride) with the
// largest record count, so no offset is range-checked away; the vector
// offset goes in as a signed int, so callers keep it below 2 GiB.
// 0x00020000 is the gfx9-family word 3 (32-bit data format).
typedef __amdgpu_buffer_rsrc_t BufRsrc;
__device__ __forceinline__ BufRsrc buf_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, -1, 0x00020000);
}
__device__ __forceinline__ void dma16(BufRsrc r, uint32_t voff, int soff, bf16_t* lds_dst) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_dst, 16, (int)voff,
                                           soff, 0, 0);
}

// ---- wavefront reductions (64 lanes) ---------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

}  // namespace sr

// ---- host-side status plumbing ----------------------------------------------
namespace sr {
struct Error {
  int status;
  std::string msg;
};
void set_error(const std::string& msg);
}  // namespace sr

#define SR_HIP(call)                                                                  \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) {                                                           \
      throw sr::Error{4, std::string("HIP error: ") + hipGetErrorString(e_) + " at " + \
                             __FILE__ + ":" + std::to_string(__LINE__) + " (" #call ")"}; \
    }                                                                                 \
  } while (0)

#define SR_CHECK_LAUNCH() SR_HIP(hipGetLastError())

// Optional timing of kernel launches by their own dispatch packets.  While
// sr::launch_timing points at a pair of events, every launch through
// SR_LAUNCH stamps the end of its kernel into `stop` (the last launch wins)
// and the first one also the start of its kernel into `start`; no marker
// packets go between the kernels.  Without it SR_LAUNCH is a plain launch.
namespace sr {
struct LaunchTiming {
  hipEvent_t start, stop;
  bool started;
};
extern thread_local LaunchTiming* launch_timing;
}  // namespace sr
#define SR_LAUNCH(kernel, grid, block, shmem, stream, ...)                                                  \
  do {                                                                                                      \
    sr::LaunchTiming* lt_ = sr::launch_timing;                                                            \
    if (lt_) {                                                                                              \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, lt_->started ? nullptr : lt_->start, lt_->stop, \
                            0, __VA_ARGS__);                                                              \
      lt_->started = true;                                                                                  \
    } else {                                                                                                \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                                  \
    }                                                                                                       \
  } while (0)

#define SR_REQUIRE(cond, code, text)                \
  do {                                              \
    if (!(cond)) throw sr::Error{(code), (text)};   \
  } while (0)
