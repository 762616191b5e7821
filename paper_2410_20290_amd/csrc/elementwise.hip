// Embedding gather, RMSNorm, RoPE (table + fused scatter into the KV cache),
// the reward model's scalar head and small helpers.
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
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, (const bf16_t*)E, d, tok, h);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)E, d, tok, h);
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

void rmsnorm(int dtype, const float* x, int ldx, const void* g, int d, float eps, int rows, void* out,
             int ldo, hipStream_t s) {
  if (rows <= 0) return;
  if (dtype == SR_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, x, ldx, (const bf16_t*)g, d,
                       eps, (bf16_t*)out, ldo);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(rows), dim3(256), 0, s, x, ldx, (const float*)g, d,
                       eps, (float*)out, ldo);
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
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks), dim3(256), 0, s, tab, npos, hd, theta);
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
    hipLaunchKernelGGL(rope_scatter_kernel<bf16_t>, grid, dim3(256), 0, s, qkv, lr, hq, hkv, hd, tab,
                       pos0, qout, (bf16_t*)kdst, (bf16_t*)vdst, cap, t0);
  else
    hipLaunchKernelGGL(rope_scatter_kernel<float>, grid, dim3(256), 0, s, qkv, lr, hq, hkv, hd, tab,
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
    hipLaunchKernelGGL(embed_norm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, (const bf16_t*)E, d, tok,
                       (const bf16_t*)g, eps, h, (bf16_t*)xn);
  else
    hipLaunchKernelGGL(embed_norm_kernel<float>, dim3(rows), dim3(256), 0, s, (const float*)E, d, tok,
                       (const float*)g, eps, h, (float*)xn);
  SR_CHECK_LAUNCH();
}

// One block per row: h += sum of split partials (in split order); xn = RMSNorm(h) * g.
// Threads own float4 column chunks; the chunks of one thread (up to 4 per
// pass) are independent, so their loads are in flight together.
template <typename T>
__global__ void __launch_bounds__(256)
add_norm_kernel(const float* __restrict__ part, int splits, int rows, int d, float* __restrict__ h,
                const T* __restrict__ g, float eps, T* __restrict__ xn) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const int d4 = d / 4;
  float4* hr = reinterpret_cast<float4*>(h + (int64_t)r * d);
  const float4* pr = reinterpret_cast<const float4*>(part + (int64_t)r * d);
  const int64_t sstride4 = (int64_t)rows * d4;
  float ss = 0.f;
  for (int base = 0; base < d4; base += 4 * 256) {
    float4 v[4];
    bool ok[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = base + u * 256 + threadIdx.x;
      ok[u] = j < d4;
      v[u] = ok[u] ? hr[j] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int sp = 0; sp < splits; ++sp) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = base + u * 256 + threadIdx.x;
        if (ok[u]) {
          const float4 p = pr[sp * sstride4 + j];
          v[u].x += p.x; v[u].y += p.y; v[u].z += p.z; v[u].w += p.w;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int j = base + u * 256 + threadIdx.x;
      if (ok[u]) {
        hr[j] = v[u];
        ss += v[u].x * v[u].x + v[u].y * v[u].y + v[u].z * v[u].z + v[u].w * v[u].w;
      }
    }
  }
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  const float* hs = h + (int64_t)r * d;
  T* o = xn + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += 256) o[i] = from_f32<T>(hs[i] * inv * to_f32<T>(g[i]));
}

// Row-parallel form for few rows: grid (rows, ceil(d / 1024)).  The first
// kernel adds the split partials into h and leaves each block's sum of
// squares; the second sums those in block order and normalises.
__global__ void __launch_bounds__(256)
add_rows_kernel(const float* __restrict__ part, int splits, int rows, int d, float* __restrict__ h,
                float* __restrict__ ssp) {
  __shared__ float red[4];
  const int r = blockIdx.x, blk = blockIdx.y, nblk = gridDim.y;
  const int d4 = d / 4;
  const int j = blk * 256 + threadIdx.x;
  float ss = 0.f;
  if (j < d4) {
    float4* hr = reinterpret_cast<float4*>(h + (int64_t)r * d);
    const float4* pr = reinterpret_cast<const float4*>(part + (int64_t)r * d);
    const int64_t sstride4 = (int64_t)rows * d4;
    float4 v = hr[j];
    for (int sp = 0; sp < splits; ++sp) {
      const float4 p = pr[sp * sstride4 + j];
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    hr[j] = v;
    ss = v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = block_sum256(ss, red);
  if (threadIdx.x == 0) ssp[(int64_t)r * nblk + blk] = ss;
}

template <typename T>
__global__ void __launch_bounds__(256)
norm_rows_kernel(const float* __restrict__ h, int d, const float* __restrict__ ssp, const T* __restrict__ g,
                 float eps, T* __restrict__ xn) {
  const int r = blockIdx.x, blk = blockIdx.y, nblk = gridDim.y;
  float ss = 0.f;
  for (int b = 0; b < nblk; ++b) ss += ssp[(int64_t)r * nblk + b];
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  const int c0 = blk * 1024, c1 = min(d, c0 + 1024);
  const float* hr = h + (int64_t)r * d;
  T* o = xn + (int64_t)r * d;
  for (int i = c0 + threadIdx.x; i < c1; i += 256) o[i] = from_f32<T>(hr[i] * inv * to_f32<T>(g[i]));
}

void add_norm(int dtype, const float* part, int splits, int rows, int d, float* h, const void* g, float eps,
              void* xn, float* ssp, hipStream_t s) {
  if (rows <= 0) return;
  SR_REQUIRE(d % 4 == 0, 3, "d_model must be a multiple of 4");
  if (ssp && rows < 256) {
    dim3 grid(rows, (d + 1023) / 1024);
    hipLaunchKernelGGL(add_rows_kernel, grid, dim3(256), 0, s, part, splits, rows, d, h, ssp);
    SR_CHECK_LAUNCH();
    if (dtype == SR_BF16)
      hipLaunchKernelGGL(norm_rows_kernel<bf16_t>, grid, dim3(256), 0, s, h, d, ssp, (const bf16_t*)g, eps,
                         (bf16_t*)xn);
    else
      hipLaunchKernelGGL(norm_rows_kernel<float>, grid, dim3(256), 0, s, h, d, ssp, (const float*)g, eps,
                         (float*)xn);
    SR_CHECK_LAUNCH();
    return;
  }
  if (dtype == SR_BF16)
    hipLaunchKernelGGL(add_norm_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, part, splits, rows, d, h,
                       (const bf16_t*)g, eps, (bf16_t*)xn);
  else
    hipLaunchKernelGGL(add_norm_kernel<float>, dim3(rows), dim3(256), 0, s, part, splits, rows, d, h,
                       (const float*)g, eps, (float*)xn);
  SR_CHECK_LAUNCH();
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
    hipLaunchKernelGGL(qkv_finalize_kernel<bf16_t>, grid, dim3(64), 0, s, part, splits, rows, hq, hkv, hd, tab,
                       pos, qout, (bf16_t*)kdst, (bf16_t*)vdst, cap, t0);
  else
    hipLaunchKernelGGL(qkv_finalize_kernel<float>, grid, dim3(64), 0, s, part, splits, rows, hq, hkv, hd, tab,
                       pos, qout, (float*)kdst, (float*)vdst, cap, t0);
  SR_CHECK_LAUNCH();
}

template <typename T>
__global__ void __launch_bounds__(256)
score_head_kernel(const float* __restrict__ h, int d, int lr, const int32_t* __restrict__ len,
                  const T* __restrict__ g, const T* __restrict__ w, float eps, float* __restrict__ score) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const float* x = h + ((int64_t)r * lr + (len[r] - 1)) * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += x[i] * x[i];
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  float dot = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) dot += (x[i] * inv * to_f32<T>(g[i])) * to_f32<T>(w[i]);
  dot = block_sum256(dot, red);
  if (threadIdx.x == 0) score[r] = dot;
}

void score_head(int dtype, const float* h, int d, int lr, const int32_t* len, int rows,
                const void* g, const void* w, float eps, float* score, hipStream_t s) {
  if (rows <= 0) return;
  if (dtype == SR_BF16)
    hipLaunchKernelGGL(score_head_kernel<bf16_t>, dim3(rows), dim3(256), 0, s, h, d, lr, len,
                       (const bf16_t*)g, (const bf16_t*)w, eps, score);
  else
    hipLaunchKernelGGL(score_head_kernel<float>, dim3(rows), dim3(256), 0, s, h, d, lr, len,
                       (const float*)g, (const float*)w, eps, score);
  SR_CHECK_LAUNCH();
}

__global__ void gather_tokens_kernel(const int32_t* __restrict__ store, int ld, const int32_t* __restrict__ cand,
                                     const int32_t* __restrict__ len, int lr, int32_t* __restrict__ tokens) {
  const int r = blockIdx.x;
  const int32_t* src = store + (int64_t)cand[r] * ld;
  const int n = len[r];
  for (int t = threadIdx.x; t < lr; t += blockDim.x) tokens[(int64_t)r * lr + t] = t < n ? src[t] : 0;
}

void gather_tokens(const int32_t* store, int ld, const int32_t* cand, const int32_t* len, int rows,
                   int lr, int32_t* tokens, hipStream_t s) {
  if (rows <= 0) return;
  hipLaunchKernelGGL(gather_tokens_kernel, dim3(rows), dim3(256), 0, s, store, ld, cand, len, lr, tokens);
  SR_CHECK_LAUNCH();
}

__global__ void philox_fill_kernel(uint2 key, const uint4* __restrict__ ctr, int n, uint4* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = philox4x32_10(ctr[i], key);
}

void philox_fill(uint64_t seed, const uint32_t* ctr, int n, uint32_t* out, hipStream_t s) {
  if (n <= 0) return;
  uint2 key = make_uint2((uint32_t)seed, (uint32_t)(seed >> 32));
  hipLaunchKernelGGL(philox_fill_kernel, dim3((n + 255) / 256), dim3(256), 0, s, key,
                     (const uint4*)ctr, n, (uint4*)out);
  SR_CHECK_LAUNCH();
}

}  // namespace sr
