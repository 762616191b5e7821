// Attention of the decoder.
//
// Decode: every candidate row has one query (the newest token).  Keys are
// the prompt prefix, stored once and shared by all rows, followed by the
// row's own tail.  A work-group owns (row, KV head, key split) and serves the
// whole query-head group of that KV head, so each K/V byte is read once per
// row.  16-byte loads; lanes of one key row are adjacent, so a wave reads
// whole contiguous rows.  Online softmax in base 2; split partials are merged
// by log-sum-exp in a second kernel.
//
// Prefill (reward-model scoring, prompt): a work-group owns a block of
// queries of one row and one KV head; K/V tiles are staged in LDS as fp32
// and shared by all its queries.
#include "common.h"
#include "kernels.h"

namespace sr {

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float exp2_or_zero(float x) { return x == -INFINITY ? 0.f : exp2f(x); }

template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
decode_attn_kernel(const float* __restrict__ q, const T* __restrict__ kpre, const T* __restrict__ vpre,
                   int P, const T* __restrict__ ktail, const T* __restrict__ vtail, int cap, int lt,
                   int hq, int hkv, int kps, int splits, float* __restrict__ part,
                   T* __restrict__ out, float qscale) {
  constexpr int EPL = Vec16<T>::N;   // elements per 16-byte load
  constexpr int LPK = HD / EPL;      // lanes per key row
  constexpr int KPW = 64 / LPK;      // keys per wave step
  constexpr int U = 4;               // keys per lane per iteration
  constexpr int NW = 4;              // waves
  const int split = blockIdx.x, h = blockIdx.y, row = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPK, ks = lane / LPK;
  const int total = P + lt;
  const int k0 = split * kps, k1 = min(total, k0 + kps);

  float qv[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < EPL; ++e)
      qv[g][e] = q[((int64_t)row * hq + h * G + g) * HD + sub * EPL + e] * qscale;

  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }
  const T* kt = ktail + ((int64_t)row * hkv + h) * cap * HD;
  const T* vt = vtail + ((int64_t)row * hkv + h) * cap * HD;
  const T* kp = kpre + (int64_t)h * P * HD;
  const T* vp = vpre + (int64_t)h * P * HD;

  for (int base = k0; base < k1; base += NW * KPW * U) {
    float kf[U][EPL], vf[U][EPL];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + (u * NW + wave) * KPW + ks;
      valid[u] = j < k1;
      if (valid[u]) {
        const T* kr = (j < P) ? kp + (int64_t)j * HD : kt + (int64_t)(j - P) * HD;
        const T* vr = (j < P) ? vp + (int64_t)j * HD : vt + (int64_t)(j - P) * HD;
        Vec16<T>::load(kr + sub * EPL, kf[u]);
        Vec16<T>::load(vr + sub * EPL, vf[u]);
      } else {
#pragma unroll
        for (int e = 0; e < EPL; ++e) kf[u][e] = vf[u][e] = 0.f;
      }
    }
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d = fmaf(qv[g][e], kf[u][e], d);
#pragma unroll
        for (int o = LPK / 2; o > 0; o >>= 1) d += __shfl_xor(d, o, 64);
        s[u][g] = valid[u] ? d : -INFINITY;
      }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mt = s[0][g];
#pragma unroll
      for (int u = 1; u < U; ++u) mt = fmaxf(mt, s[u][g]);
      const float mn = fmaxf(m[g], mt);
      if (mn == -INFINITY) continue;
      const float corr = exp2_or_zero(m[g] - mn);
      l[g] *= corr;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] *= corr;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2_or_zero(s[u][g] - mn);
        l[g] += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[u][e], acc[g][e]);
      }
      m[g] = mn;
    }
  }

  // merge the KPW key slots of a wave (lanes with equal `sub`)
#pragma unroll
  for (int o = LPK; o < 64; o <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mo = __shfl_xor(m[g], o, 64);
      const float lo = __shfl_xor(l[g], o, 64);
      const float mn = fmaxf(m[g], mo);
      const float c1 = (mn == -INFINITY) ? 0.f : exp2_or_zero(m[g] - mn);
      const float c2 = (mn == -INFINITY) ? 0.f : exp2_or_zero(mo - mn);
      l[g] = l[g] * c1 + lo * c2;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const float ao = __shfl_xor(acc[g][e], o, 64);
        acc[g][e] = acc[g][e] * c1 + ao * c2;
      }
      m[g] = mn;
    }
  }
  // merge the waves through LDS
  __shared__ float sm[NW][G], sl[NW][G];
  __shared__ float sacc[NW][G][HD];
  if (ks == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (sub == 0) {
        sm[wave][g] = m[g];
        sl[wave][g] = l[g];
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) sacc[wave][g][sub * EPL + e] = acc[g][e];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * HD; idx += blockDim.x) {
    const int g = idx / HD, dd = idx % HD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm[w][g]);
    float L = 0.f, A = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float c = exp2_or_zero(sm[w][g] - M);
        L += sl[w][g] * c;
        A += sacc[w][g][dd] * c;
      }
    }
    const int qh = h * G + g;
    if (splits == 1) {
      out[((int64_t)row * hq + qh) * HD + dd] = from_f32<T>(A / L);
    } else {
      float* p = part + (((int64_t)row * hq + qh) * splits + split) * (HD + 2);
      p[dd] = A;
      if (dd == 0) {
        p[HD] = M;
        p[HD + 1] = L;
      }
    }
  }
}

template <typename T, int HD>
__global__ void decode_merge_kernel(const float* __restrict__ part, int splits, int hq,
                                    T* __restrict__ out) {
  const int rq = blockIdx.x;  // row * hq + qh
  const float* p = part + (int64_t)rq * splits * (HD + 2);
  float M = -INFINITY;
  for (int s = 0; s < splits; ++s) M = fmaxf(M, p[s * (HD + 2) + HD]);
  for (int dd = threadIdx.x; dd < HD; dd += blockDim.x) {
    float L = 0.f, A = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float c = exp2_or_zero(p[s * (HD + 2) + HD] - M);
      L += p[s * (HD + 2) + HD + 1] * c;
      A += p[s * (HD + 2) + dd] * c;
    }
    out[(int64_t)rq * HD + dd] = from_f32<T>(A / L);
  }
}

// Keys per split: aim for enough work-groups to fill the chip, at least 256
// keys per split.
static int decode_kps(int rows, int hkv, int keys) {
  int64_t groups = (int64_t)rows * hkv;
  int splits = 1;
  while (groups * splits < 1024 && keys / (splits * 2) >= 256) splits *= 2;
  return (keys + splits - 1) / splits;
}

int decode_attn_splits(int rows, int hkv, int keys) {
  int kps = decode_kps(rows, hkv, keys);
  return (keys + kps - 1) / kps;
}

template <typename T, int HD, int G>
static void launch_decode(const DecodeAttnArgs& a, hipStream_t s) {
  const int keys = a.P + a.lt;
  const int kps = decode_kps(a.rows, a.hkv, keys);
  const int splits = (keys + kps - 1) / kps;
  if (splits > 1)
    SR_REQUIRE((size_t)a.rows * a.hq * splits * (HD + 2) <= a.part_cap, 5,
               "attention partial buffer too small");
  const float qscale = kLog2e / sqrtf((float)HD);
  hipLaunchKernelGGL((decode_attn_kernel<T, HD, G>), dim3(splits, a.hkv, a.rows), dim3(256), 0, s,
                     a.q, (const T*)a.kpre, (const T*)a.vpre, a.P, (const T*)a.ktail,
                     (const T*)a.vtail, a.cap, a.lt, a.hq, a.hkv, kps, splits, a.part, (T*)a.out,
                     qscale);
  SR_CHECK_LAUNCH();
  if (splits > 1) {
    hipLaunchKernelGGL((decode_merge_kernel<T, HD>), dim3(a.rows * a.hq), dim3(HD), 0, s, a.part,
                       splits, a.hq, (T*)a.out);
    SR_CHECK_LAUNCH();
  }
}

template <typename T, int HD>
static void decode_by_group(const DecodeAttnArgs& a, hipStream_t s) {
  switch (a.hq / a.hkv) {
    case 1: launch_decode<T, HD, 1>(a, s); break;
    case 2: launch_decode<T, HD, 2>(a, s); break;
    case 4: launch_decode<T, HD, 4>(a, s); break;
    case 8: launch_decode<T, HD, 8>(a, s); break;
    default: SR_REQUIRE(false, 3, "query heads per KV head must be 1, 2, 4 or 8");
  }
}

template <typename T>
static void decode_by_hd(const DecodeAttnArgs& a, hipStream_t s) {
  switch (a.hd) {
    case 32: decode_by_group<T, 32>(a, s); break;
    case 64: decode_by_group<T, 64>(a, s); break;
    case 128: decode_by_group<T, 128>(a, s); break;
    default: SR_REQUIRE(false, 3, "head_dim must be 32, 64 or 128");
  }
}

void decode_attn(const DecodeAttnArgs& a, hipStream_t s) {
  if (a.rows <= 0) return;
  if (a.dtype == SR_BF16) decode_by_hd<bf16_t>(a, s);
  else decode_by_hd<float>(a, s);
}

// --------------------------------------------------------------- prefill
// 256 threads = QB queries x G heads x 4 threads; thread `sub` of a
// (query, head) pair owns dimensions sub, sub + 4, sub + 8, ...
template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
prefill_attn_kernel(const float* __restrict__ q, const T* __restrict__ kpre, const T* __restrict__ vpre,
                    int P, const T* __restrict__ kown, const T* __restrict__ vown, int lr, int hq,
                    int hkv, T* __restrict__ out, float qscale) {
  constexpr int TPQ = 4, DPT = HD / TPQ, QB = 64 / G, KT = 32;
  constexpr int EPL = Vec16<T>::N, CPR = HD / EPL;
  __shared__ float Ks[KT][HD];
  __shared__ float Vs[KT][HD];
  const int qb = blockIdx.x, h = blockIdx.y, row = blockIdx.z;
  const int tid = threadIdx.x;
  const int sub = tid % TPQ, pair = tid / TPQ, g = pair % G, qi = pair / G;
  const int t = qb * QB + qi;
  const bool qvalid = t < lr;
  const int qh = h * G + g;
  float qv[DPT], acc[DPT];
#pragma unroll
  for (int d = 0; d < DPT; ++d) {
    qv[d] = qvalid ? q[(((int64_t)row * lr + t) * hq + qh) * HD + d * TPQ + sub] * qscale : 0.f;
    acc[d] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int tlast = min(lr, (qb + 1) * QB) - 1;
  const int nkeys = P + tlast + 1;
  const T* kp = kpre + (int64_t)h * P * HD;
  const T* vp = vpre + (int64_t)h * P * HD;
  const T* ko = kown + ((int64_t)row * hkv + h) * lr * HD;
  const T* vo = vown + ((int64_t)row * hkv + h) * lr * HD;
  for (int kb = 0; kb < nkeys; kb += KT) {
    for (int idx = tid; idx < KT * CPR; idx += 256) {
      const int j = idx / CPR, c = idx % CPR;
      const int key = kb + j;
      float kf[EPL], vf[EPL];
      if (key < nkeys) {
        const T* kr = key < P ? kp + (int64_t)key * HD : ko + (int64_t)(key - P) * HD;
        const T* vr = key < P ? vp + (int64_t)key * HD : vo + (int64_t)(key - P) * HD;
        Vec16<T>::load(kr + c * EPL, kf);
        Vec16<T>::load(vr + c * EPL, vf);
      } else {
#pragma unroll
        for (int e = 0; e < EPL; ++e) kf[e] = vf[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        Ks[j][c * EPL + e] = kf[e];
        Vs[j][c * EPL + e] = vf[e];
      }
    }
    __syncthreads();
    float s[KT];
    float mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      float d = 0.f;
#pragma unroll
      for (int dd = 0; dd < DPT; ++dd) d = fmaf(qv[dd], Ks[j][dd * TPQ + sub], d);
      d += __shfl_xor(d, 1, 64);
      d += __shfl_xor(d, 2, 64);
      const int key = kb + j;
      const bool ok = qvalid && key <= P + t;
      s[j] = ok ? d : -INFINITY;
      mt = fmaxf(mt, s[j]);
    }
    const float mn = fmaxf(m, mt);
    if (mn != -INFINITY) {
      const float corr = exp2_or_zero(m - mn);
      l *= corr;
#pragma unroll
      for (int dd = 0; dd < DPT; ++dd) acc[dd] *= corr;
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        const float p = exp2_or_zero(s[j] - mn);
        l += p;
#pragma unroll
        for (int dd = 0; dd < DPT; ++dd) acc[dd] = fmaf(p, Vs[j][dd * TPQ + sub], acc[dd]);
      }
      m = mn;
    }
    __syncthreads();
  }
  if (qvalid) {
    T* o = out + (((int64_t)row * lr + t) * hq + qh) * HD;
#pragma unroll
    for (int dd = 0; dd < DPT; ++dd) o[dd * TPQ + sub] = from_f32<T>(acc[dd] / l);
  }
}

template <typename T, int HD, int G>
static void launch_prefill(const PrefillAttnArgs& a, hipStream_t s) {
  constexpr int QB = 64 / G;
  const float qscale = kLog2e / sqrtf((float)HD);
  dim3 grid((a.lr + QB - 1) / QB, a.hkv, a.rows);
  hipLaunchKernelGGL((prefill_attn_kernel<T, HD, G>), grid, dim3(256), 0, s, a.q, (const T*)a.kpre,
                     (const T*)a.vpre, a.P, (const T*)a.kown, (const T*)a.vown, a.lr, a.hq, a.hkv,
                     (T*)a.out, qscale);
  SR_CHECK_LAUNCH();
}

template <typename T, int HD>
static void prefill_by_group(const PrefillAttnArgs& a, hipStream_t s) {
  switch (a.hq / a.hkv) {
    case 1: launch_prefill<T, HD, 1>(a, s); break;
    case 2: launch_prefill<T, HD, 2>(a, s); break;
    case 4: launch_prefill<T, HD, 4>(a, s); break;
    case 8: launch_prefill<T, HD, 8>(a, s); break;
    default: SR_REQUIRE(false, 3, "query heads per KV head must be 1, 2, 4 or 8");
  }
}

template <typename T>
static void prefill_by_hd(const PrefillAttnArgs& a, hipStream_t s) {
  switch (a.hd) {
    case 32: prefill_by_group<T, 32>(a, s); break;
    case 64: prefill_by_group<T, 64>(a, s); break;
    case 128: prefill_by_group<T, 128>(a, s); break;
    default: SR_REQUIRE(false, 3, "head_dim must be 32, 64 or 128");
  }
}

void prefill_attn(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.rows <= 0 || a.lr <= 0) return;
  if (a.dtype == SR_BF16) prefill_by_hd<bf16_t>(a, s);
  else prefill_by_hd<float>(a, s);
}

}  // namespace sr
