// Embedding gather, RMSNorm, RoPE (table + fused scatter into the KV cache),
// the reward model's scalar head and small helpers.
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "philox.h"

namespace sr {

template <typename T>
__global__ void embed_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ tok,
                             float* __restrict__ h) {
  const int r = blockIdx.x;
  const T* src = E + (int64_t)tok[r] * d;
  float* dst = h + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) dst[i] = to_f32<T>(src[i]);
}

void embed(int dtype, const void* E, int d, const int32_t* tok, int rows, float* h, hipStream_t s) {
  if (rows <= 0) return;
  if (dtype == SR_BF16)
    SR_LAUNCH(embed_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, (const bf16_t*)E, d, tok, h);
  else
    SR_LAUNCH(embed_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)E, d, tok, h);
  SR_CHECK_LAUNCH();
}

// Block-wide sum over 256 threads.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float t = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return t;
}

template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x, int ldx,
                                                      const T* __restrict__ g, int d, float eps,
                                                      T* __restrict__ out, int ldo) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const float* xr = x + (int64_t)r * ldx;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += xr[i] * xr[i];
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  T* o = out + (int64_t)r * ldo;
  for (int i = threadIdx.x; i < d; i += 256) o[i] = from_f32<T>(xr[i] * inv * to_f32<T>(g[i]));
}

// Four consecutive elements of T.
__device__ __forceinline__ float4 load4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 load4(const bf16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u), __uint_as_float(u.y << 16),
                     __uint_as_float(u.y & 0xFFFF0000u));
}
__device__ __forceinline__ void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4(bf16_t* p, float4 v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16),
                                            f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16));
}

// Rows whose width is a multiple of 4 and at most 256 KV float4s: the row
// is loaded once as float4s (all loads in flight together), kept in
// registers for the scaling pass, and written four elements per store.
template <typename T, int KV>
__global__ void __launch_bounds__(256) rmsnorm_vec_kernel(const float* __restrict__ x, int ldx,
                                                          const T* __restrict__ g, int d, float eps,
                                                          T* __restrict__ out, int ldo) {
  __shared__ float red[4];
  const int r = blockIdx.x, d4 = d / 4;
  const float* xr = x + (int64_t)r * ldx;
  float4 v[KV];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < KV; ++k) {
    const int j = threadIdx.x + 256 * k;
    v[k] = j < d4 ? load4(xr + 4 * j) : make_float4(0.f, 0.f, 0.f, 0.f);
    ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  }
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  T* o = out + (int64_t)r * ldo;
#pragma unroll
  for (int k = 0; k < KV; ++k) {
    const int j = threadIdx.x + 256 * k;
    if (j >= d4) continue;
    const float4 w = load4(g + 4 * j);
    store4(o + 4 * j, make_float4(v[k].x * inv * w.x, v[k].y * inv * w.y, v[k].z * inv * w.z, v[k].w * inv * w.w));
  }
}

void rmsnorm(int dtype, const float* x, int ldx, const void* g, int d, float eps, int rows, void* out,
             int ldo, hipStream_t s) {
  if (rows <= 0) return;
  const bool vec = d % 4 == 0 && ldx % 4 == 0 && ldo % 4 == 0 && d <= 4 * 256 * 4 &&
                   (reinterpret_cast<uintptr_t>(x) & 15) == 0 && (reinterpret_cast<uintptr_t>(out) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(g) & 15) == 0;
  const int kv = (d / 4 + 255) / 256;
#define SR_NORM(T, KV)                                                                                     \
  SR_LAUNCH((rmsnorm_vec_kernel<T, KV>), dim3(rows), dim3(256), 0, s, x, ldx, (const T*)g, d, eps, \
                     (T*)out, ldo)
  if (vec && dtype == SR_BF16) {
    if (kv <= 1) SR_NORM(bf16_t, 1);
    else if (kv <= 2) SR_NORM(bf16_t, 2);
    else SR_NORM(bf16_t, 4);
  } else if (vec) {
    if (kv <= 1) SR_NORM(float, 1);
    else if (kv <= 2) SR_NORM(float, 2);
    else SR_NORM(float, 4);
  } else if (dtype == SR_BF16) {
    SR_LAUNCH(rmsnorm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, x, ldx, (const bf16_t*)g, d,
                       eps, (bf16_t*)out, ldo);
  } else {
    SR_LAUNCH(rmsnorm_kernel<float>, dim3(rows), dim3(256), 0, s, x, ldx, (const float*)g, d,
                       eps, (float*)out, ldo);
  }
#undef SR_NORM
  SR_CHECK_LAUNCH();
}

__global__ void rope_table_kernel(float2* tab, int npos, int hd, double theta) {
  const int half = hd / 2;
  const int64_t total = (int64_t)npos * half;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int p = (int)(idx / half), i = (int)(idx % half);
    const double freq = pow(theta, -2.0 * (double)i / (double)hd);
    const double ang = (double)p * freq;
    tab[idx] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

void rope_table(float2* tab, int npos, int hd, double theta, hipStream_t s) {
  int64_t total = (int64_t)npos * (hd / 2);
  int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
  SR_LAUNCH(rope_table_kernel, dim3(blocks), dim3(256), 0, s, tab, npos, hd, theta);
  SR_CHECK_LAUNCH();
}

// One block per token.  Threads first rotate q and k pairs, then copy v.
template <typename T>
__global__ void __launch_bounds__(256)
rope_scatter_kernel(const float* __restrict__ qkv, int lr, int hq, int hkv, int hd,
                    const float2* __restrict__ tab, int pos0, float* __restrict__ qout,
                    T* __restrict__ kdst, T* __restrict__ vdst, int cap, int t0) {
  const int tokidx = blockIdx.x;
  const int r = tokidx / lr, t = tokidx % lr;
  const int half = hd / 2;
  const int qkv_dim = (hq + 2 * hkv) * hd;
  const float* src = qkv + (int64_t)tokidx * qkv_dim;
  const float2* cs = tab + (int64_t)(pos0 + t) * half;
  // rotations: (hq + hkv) heads x half pairs
  for (int idx = threadIdx.x; idx < (hq + hkv) * half; idx += blockDim.x) {
    const int head = idx / half, i = idx % half;
    const float x1 = src[head * hd + i], x2 = src[head * hd + half + i];
    const float2 c = cs[i];
    const float y1 = x1 * c.x - x2 * c.y;
    const float y2 = x2 * c.x + x1 * c.y;
    if (head < hq) {
      float* qo = qout + ((int64_t)tokidx * hq + head) * hd;
      qo[i] = y1;
      qo[half + i] = y2;
    } else {
      const int kh = head - hq;
      T* ko = kdst + (((int64_t)r * hkv + kh) * cap + t0 + t) * hd;
      ko[i] = from_f32<T>(y1);
      ko[half + i] = from_f32<T>(y2);
    }
  }
  for (int idx = threadIdx.x; idx < hkv * hd; idx += blockDim.x) {
    const int kh = idx / hd, i = idx % hd;
    T* vo = vdst + (((int64_t)r * hkv + kh) * cap + t0 + t) * hd;
    vo[i] = from_f32<T>(src[(hq + hkv) * hd + kh * hd + i]);
  }
}

void rope_scatter(int dtype, const float* qkv, int rows, int lr, int hq, int hkv, int hd,
                  const float2* tab, int pos0, float* qout, void* kdst, void* vdst, int cap,
                  int t0, hipStream_t s) {
  if (rows <= 0 || lr <= 0) return;
  dim3 grid(rows * lr);
  if (dtype == SR_BF16)
    SR_LAUNCH(rope_scatter_kernel<bf16_t>, grid, dim3(256), 0, s, qkv, lr, hq, hkv, hd, tab,
                       pos0, qout, (bf16_t*)kdst, (bf16_t*)vdst, cap, t0);
  else
    SR_LAUNCH(rope_scatter_kernel<float>, grid, dim3(256), 0, s, qkv, lr, hq, hkv, hd, tab,
                       pos0, qout, (float*)kdst, (float*)vdst, cap, t0);
  SR_CHECK_LAUNCH();
}

// One block per row: h = E[tok]; xn = RMSNorm(h) * g.
template <typename T>
__global__ void __launch_bounds__(256)
embed_norm_kernel(const T* __restrict__ E, int d, const int32_t* __restrict__ tok, const T* __restrict__ g,
                  float eps, float* __restrict__ h, T* __restrict__ xn) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const T* src = E + (int64_t)tok[r] * d;
  float* hr = h + (int64_t)r * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = to_f32<T>(src[i]);
    hr[i] = v;
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  T* o = xn + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += 256) o[i] = from_f32<T>(hr[i] * inv * to_f32<T>(g[i]));
}

void embed_norm(int dtype, const void* E, int d, const int32_t* tok, int rows, const void* g, float eps,
                float* h, void* xn, hipStream_t s) {
  if (rows <= 0) return;
  if (dtype == SR_BF16)
    SR_LAUNCH(embed_norm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, (const bf16_t*)E, d, tok,
                       (const bf16_t*)g, eps, h, (bf16_t*)xn);
  else
    SR_LAUNCH(embed_norm_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)E, d, tok,
                       (const float*)g, eps, h, (float*)xn);
  SR_CHECK_LAUNCH();
}

// One block per row: h += sum of split partials (in split order); xn =
// RMSNorm(h) * g.  Up to 1024 threads, each owning KV float4 chunks of the
// row; the row and all its partials are loaded at once (the partial loads
// of up to 8 splits are issued together and added in split order), the new
// h stays in registers for the normalisation.
template <typename T, int KV>
__global__ void __launch_bounds__(1024)
add_norm_kernel(const float* __restrict__ part, int splits, int rows, int d, float* __restrict__ h,
                const T* __restrict__ g, float eps, T* __restrict__ xn) {
  __shared__ float red[16];
  const int r = blockIdx.x, nt = blockDim.x, tid = threadIdx.x;
  const int d4 = d / 4;
  float4* hr = reinterpret_cast<float4*>(h + (int64_t)r * d);
  const float4* pr = reinterpret_cast<const float4*>(part + (int64_t)r * d);
  const int64_t sstride4 = (int64_t)rows * d4;
  float4 v[KV];
  bool ok[KV];
#pragma unroll
  for (int k = 0; k < KV; ++k) {
    const int j = tid + k * nt;
    ok[k] = j < d4;
    v[k] = hr[ok[k] ? j : 0];
  }
  for (int s0 = 0; s0 < splits; s0 += 8) {
    float4 p[8][KV];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int k = 0; k < KV; ++k) {
        const int j = ok[k] ? tid + k * nt : 0;
        p[u][k] = s0 + u < splits ? pr[(s0 + u) * sstride4 + j] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int k = 0; k < KV; ++k)
        if (s0 + u < splits) {
          v[k].x += p[u][k].x; v[k].y += p[u][k].y; v[k].z += p[u][k].z; v[k].w += p[u][k].w;
        }
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < KV; ++k)
    if (ok[k]) ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  // block sum in a fixed order: waves, then the wave totals in wave order
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
  for (int w = 0; w < (nt >> 6); ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  T* o = xn + (int64_t)r * d;
#pragma unroll
  for (int k = 0; k < KV; ++k) {
    if (!ok[k]) continue;
    const int j = tid + k * nt;
    hr[j] = v[k];
    const int c = 4 * j;
    o[c] = from_f32<T>(v[k].x * inv * to_f32<T>(g[c]));
    o[c + 1] = from_f32<T>(v[k].y * inv * to_f32<T>(g[c + 1]));
    o[c + 2] = from_f32<T>(v[k].z * inv * to_f32<T>(g[c + 2]));
    o[c + 3] = from_f32<T>(v[k].w * inv * to_f32<T>(g[c + 3]));
  }
}

template <typename T>
static void launch_add_norm(const float* part, int splits, int rows, int d, float* h, const void* g, float eps,
                            void* xn, hipStream_t s) {
  const int d4 = d / 4;
  const int nt = std::min(1024, (d4 + 63) / 64 * 64);
  const int kv = (d4 + nt - 1) / nt;
  SR_REQUIRE(kv <= 4, 3, "d_model too large for add_norm");
  if (kv == 1)
    SR_LAUNCH((add_norm_kernel<T, 1>), dim3(rows), dim3(nt), 0, s, part, splits, rows, d, h,
                       (const T*)g, eps, (T*)xn);
  else if (kv == 2)
    SR_LAUNCH((add_norm_kernel<T, 2>), dim3(rows), dim3(nt), 0, s, part, splits, rows, d, h,
                       (const T*)g, eps, (T*)xn);
  else
    SR_LAUNCH((add_norm_kernel<T, 4>), dim3(rows), dim3(nt), 0, s, part, splits, rows, d, h,
                       (const T*)g, eps, (T*)xn);
  SR_CHECK_LAUNCH();
}

void add_norm(int dtype, const float* part, int splits, int rows, int d, float* h, const void* g, float eps,
              void* xn, hipStream_t s) {
  if (rows <= 0) return;
  SR_REQUIRE(d % 4 == 0, 3, "d_model must be a multiple of 4");
  if (dtype == SR_BF16) launch_add_norm<bf16_t>(part, splits, rows, d, h, g, eps, xn, s);
  else launch_add_norm<float>(part, splits, rows, d, h, g, eps, xn, s);
}

// Grid (rows, hq + 2 hkv), one wave per (row, head): sum the split partials
// of the head, rotate q and k heads, scatter.
template <typename T>
__global__ void __launch_bounds__(64)
qkv_finalize_kernel(const float* __restrict__ part, int splits, int rows, int hq, int hkv, int hd,
                    const float2* __restrict__ tab, int pos, float* __restrict__ qout, T* __restrict__ kdst,
                    T* __restrict__ vdst, int cap, int t0) {
  const int r = blockIdx.x, head = blockIdx.y;
  const int qkv_dim = (hq + 2 * hkv) * hd;
  const int64_t sstride = (int64_t)rows * qkv_dim;
  const float* src = part + (int64_t)r * qkv_dim + head * hd;
  const int half = hd / 2;
  if (head < hq + hkv) {
    const float2* cs = tab + (int64_t)pos * half;
    for (int i = threadIdx.x; i < half; i += 64) {
      float x1 = 0.f, x2 = 0.f;
      for (int sp = 0; sp < splits; ++sp) {
        x1 += src[sp * sstride + i];
        x2 += src[sp * sstride + half + i];
      }
      const float2 c = cs[i];
      const float y1 = x1 * c.x - x2 * c.y;
      const float y2 = x2 * c.x + x1 * c.y;
      if (head < hq) {
        float* qo = qout + ((int64_t)r * hq + head) * hd;
        qo[i] = y1;
        qo[half + i] = y2;
      } else {
        T* ko = kdst + (((int64_t)r * hkv + (head - hq)) * cap + t0) * hd;
        ko[i] = from_f32<T>(y1);
        ko[half + i] = from_f32<T>(y2);
      }
    }
  } else {
    T* vo = vdst + (((int64_t)r * hkv + (head - hq - hkv)) * cap + t0) * hd;
    for (int i = threadIdx.x; i < hd; i += 64) {
      float x = 0.f;
      for (int sp = 0; sp < splits; ++sp) x += src[sp * sstride + i];
      vo[i] = from_f32<T>(x);
    }
  }
}

void qkv_finalize(int dtype, const float* part, int splits, int rows, int hq, int hkv, int hd,
                  const float2* tab, int pos, float* qout, void* kdst, void* vdst, int cap, int t0,
                  hipStream_t s) {
  if (rows <= 0) return;
  dim3 grid(rows, hq + 2 * hkv);
  if (dtype == SR_BF16)
    SR_LAUNCH(qkv_finalize_kernel<bf16_t>, grid, dim3(64), 0, s, part, splits, rows, hq, hkv, hd, tab,
                       pos, qout, (bf16_t*)kdst, (bf16_t*)vdst, cap, t0);
  else
    SR_LAUNCH(qkv_finalize_kernel<float>, grid, dim3(64), 0, s, part, splits, rows, hq, hkv, hd, tab,
                       pos, qout, (float*)kdst, (float*)vdst, cap, t0);
  SR_CHECK_LAUNCH();
}

template <typename T>
__global__ void __launch_bounds__(256)
score_head_kernel(const float* __restrict__ h, int d, int lr, int t0, const int32_t* __restrict__ len,
                  const T* __restrict__ g, const T* __restrict__ w, float eps, float* __restrict__ score) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  // the caller guarantees t0 < len[r] <= t0 + lr; the clamp only keeps the
  // read inside this row's block
  const int t = min(max(len[r] - 1 - t0, 0), lr - 1);
  const float* x = h + ((int64_t)r * lr + t) * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += x[i] * x[i];
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  float dot = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) dot += (x[i] * inv * to_f32<T>(g[i])) * to_f32<T>(w[i]);
  dot = block_sum256(dot, red);
  if (threadIdx.x == 0) score[r] = dot;
}

void score_head(int dtype, const float* h, int d, int lr, int t0, const int32_t* len, int rows,
                const void* g, const void* w, float eps, float* score, hipStream_t s) {
  if (rows <= 0) return;
  if (dtype == SR_BF16)
    SR_LAUNCH(score_head_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, h, d, lr, t0, len,
                       (const bf16_t*)g, (const bf16_t*)w, eps, score);
  else
    SR_LAUNCH(score_head_kernel<float>, dim3(rows), dim3(256), 0, s, h, d, lr, t0, len,
                       (const float*)g, (const float*)w, eps, score);
  SR_CHECK_LAUNCH();
}

__global__ void gather_tokens_kernel(const int32_t* __restrict__ store, int ld, const int32_t* __restrict__ cand,
                                     const int32_t* __restrict__ len, int t0, int lr,
                                     int32_t* __restrict__ tokens) {
  const int r = blockIdx.x;
  const int32_t* src = store + (int64_t)cand[r] * ld;
  const int n = len[r];
  for (int t = threadIdx.x; t < lr; t += blockDim.x)
    tokens[(int64_t)r * lr + t] = t0 + t < n ? src[t0 + t] : 0;
}

void gather_tokens(const int32_t* store, int ld, const int32_t* cand, const int32_t* len, int rows,
                   int t0, int lr, int32_t* tokens, hipStream_t s) {
  if (rows <= 0) return;
  SR_LAUNCH(gather_tokens_kernel, dim3(rows), dim3(256), 0, s, store, ld, cand, len, t0, lr, tokens);
  SR_CHECK_LAUNCH();
}

__global__ void philox_fill_kernel(uint2 key, const uint4* __restrict__ ctr, int n, uint4* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = philox4x32_10(ctr[i], key);
}

void philox_fill(uint64_t seed, const uint32_t* ctr, int n, uint32_t* out, hipStream_t s) {
  if (n <= 0) return;
  uint2 key = make_uint2((uint32_t)seed, (uint32_t)(seed >> 32));
  SR_LAUNCH(philox_fill_kernel, dim3((n + 255) / 256), dim3(256), 0, s, key,
                     (const uint4*)ctr, n, (uint4*)out);
  SR_CHECK_LAUNCH();
}

}  // namespace sr
