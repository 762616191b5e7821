// Next-token draw (eq. auto-regressive, section 3) fused with the per-row
// state update of the generation loop.
//
// The draw is an exact integer inverse CDF so that it is a function of the
// logits alone:  m = max l;  z_i = (l_i - m) * (1/T);  p_i = exp_sr(z_i);
// w_i = trunc(p_i * 2^32) (uint64);  W = sum w_i;  x = word 0 of
// Philox4x32-10((step, cand, 0, 0), seed);  t = floor(x W / 2^32);
// token = min{i : w_0 + ... + w_i > t}.  Integer sums make the result
// independent of the reduction order.  A row without positive weight (all
// logits -inf or NaN) yields token 0.
//
// exp_sr: Cody-Waite range reduction (Cody & Waite, Software Manual for the
// Elementary Functions, 1980) with n = rint(z log2 e), r = z - n ln2_hi -
// n ln2_lo, then the degree-7 Taylor polynomial of e^r by Horner's rule and
// a scaling by 2^n.  Each step is a separately rounded float32 operation
// (this file is built with contraction off); inputs below -24 give 0.
#include "common.h"
#include "kernels.h"
#include "philox.h"

#pragma clang fp contract(off)

namespace sr {

__device__ __forceinline__ float exp_sr(float z) {
  const float kLog2e = __uint_as_float(0x3FB8AA3Bu);
  const float kLn2Hi = __uint_as_float(0x3F317200u);
  const float kLn2Lo = __uint_as_float(0x35BFBE8Eu);
  const float c2 = 0.5f, c3 = __uint_as_float(0x3E2AAAABu), c4 = __uint_as_float(0x3D2AAAABu),
              c5 = __uint_as_float(0x3C088889u), c6 = __uint_as_float(0x3AB60B61u),
              c7 = __uint_as_float(0x39500D01u);
  if (!(z >= -24.0f)) return 0.0f;  // below the cutoff, -inf and NaN
  const float n = rintf(__fmul_rn(z, kLog2e));
  float r = __fsub_rn(z, __fmul_rn(n, kLn2Hi));
  r = __fsub_rn(r, __fmul_rn(n, kLn2Lo));
  float p = c7;
  p = __fadd_rn(__fmul_rn(p, r), c6);
  p = __fadd_rn(__fmul_rn(p, r), c5);
  p = __fadd_rn(__fmul_rn(p, r), c4);
  p = __fadd_rn(__fmul_rn(p, r), c3);
  p = __fadd_rn(__fmul_rn(p, r), c2);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  p = __fadd_rn(__fmul_rn(p, r), 1.0f);
  return ldexpf(p, (int)n);
}

__device__ __forceinline__ uint64_t weight_of(float l, float m, float inv_t) {
  const float z = __fmul_rn(__fsub_rn(l, m), inv_t);
  const float p = exp_sr(z);
  return (uint64_t)__fmul_rn(p, 4294967296.0f);
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl_xor(lo, o, 64);
  hi = __shfl_xor(hi, o, 64);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_up_u64(uint64_t v, int o) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl_up(lo, o, 64);
  hi = __shfl_up(hi, o, 64);
  return ((uint64_t)hi << 32) | lo;
}

constexpr int kSampleThreads = 1024;
constexpr int kPerLane = 8;                       // consecutive elements per lane and step
constexpr int kSegment = 64 * kPerLane;           // elements per segment (one wave step)
constexpr int kMaxSegments = kSampleThreads;      // vocab <= 524288

// One work-group per row.  Pass 1: maximum and its first index.  Pass 2:
// exact integer weights, summed per segment of 512 consecutive entries (a
// wave step: 8 consecutive entries per lane, one wave reduction).  Block
// scan of the segment sums, the segment holding the drawn point, then
// wave 0 finds the lane and the lane its entry.  All sums are exact 64-bit
// integers, so the drawn token does not depend on the grouping.
__global__ void __launch_bounds__(kSampleThreads)
sample_kernel(const float* __restrict__ logits, int64_t row_stride, int vocab,
              const int32_t* __restrict__ cand, int step, float inv_t, int greedy, uint2 key,
              int32_t* __restrict__ next_tok, int32_t* __restrict__ done, int32_t* __restrict__ len,
              int32_t* __restrict__ store, int store_ld, int eos_id) {
  __shared__ uint64_t segsum[kMaxSegments];
  __shared__ float red_v[kSampleThreads / 64];
  __shared__ int red_i[kSampleThreads / 64];
  __shared__ uint64_t wave_tot[kSampleThreads / 64];
  __shared__ int found_seg;
  __shared__ uint64_t found_base;

  const int r = blockIdx.x;
  if (done && done[r]) return;  // uniform per block
  const float* lg = logits + (int64_t)r * row_stride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int NW = kSampleThreads / 64;
  if (tid == 0) {  // defaults keep every later access in bounds
    found_seg = 0;
    found_base = 0;
  }

  // 8 consecutive logits from `base` (-inf past the end); one 32-byte load
  // when the row is 16-byte aligned and the chunk is whole
  const bool vec = (reinterpret_cast<uintptr_t>(lg) & 15) == 0;
  auto load8 = [&](int base, float (&v)[kPerLane]) {
    if (vec && base + kPerLane <= vocab) {
      const float4 a = *reinterpret_cast<const float4*>(lg + base);
      const float4 b = *reinterpret_cast<const float4*>(lg + base + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
      v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
      for (int e = 0; e < kPerLane; ++e) v[e] = base + e < vocab ? lg[base + e] : -INFINITY;
    }
  };

  // pass 1: maximum (and its first index, for greedy decoding); the next
  // chunk is loaded before the current one is compared
  float mv = -INFINITY;
  int mi = 0x7FFFFFFF;
  {
    constexpr int STRIDE = kPerLane * kSampleThreads;
    float cur[kPerLane], nxt[kPerLane];
    int base = kPerLane * tid;
    load8(base, cur);
    for (; base < vocab; base += STRIDE) {
      load8(base + STRIDE, nxt);
#pragma unroll
      for (int e = 0; e < kPerLane; ++e)
        if (cur[e] > mv) { mv = cur[e]; mi = base + e; }
#pragma unroll
      for (int e = 0; e < kPerLane; ++e) cur[e] = nxt[e];
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(mv, o, 64);
    const int oi = __shfl_xor(mi, o, 64);
    if (ov > mv || (ov == mv && oi < mi)) { mv = ov; mi = oi; }
  }
  if (lane == 0) { red_v[wave] = mv; red_i[wave] = mi; }
  __syncthreads();
  float m = red_v[0];
  int am = red_i[0];
  for (int w = 1; w < NW; ++w)
    if (red_v[w] > m || (red_v[w] == m && red_i[w] < am)) { m = red_v[w]; am = red_i[w]; }

  int token;
  if (greedy) {
    token = am < vocab ? am : 0;
  } else {
    // pass 2: segment sums
    const int nseg = (vocab + kSegment - 1) / kSegment;
    {
      float cur[kPerLane], nxt[kPerLane];
      load8(wave * kSegment + kPerLane * lane, cur);
      for (int seg = wave; seg < nseg; seg += NW) {
        const int base = seg * kSegment + kPerLane * lane;
        load8(base + NW * kSegment, nxt);
        uint64_t w = 0;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) w += weight_of(cur[e], m, inv_t);  // -inf weighs 0
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) w += shfl_xor_u64(w, o);
        if (lane == 0) segsum[seg] = w;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) cur[e] = nxt[e];
      }
    }
    __syncthreads();
    // exclusive scan of the segment sums: thread t owns segment t
    const uint64_t mine = tid < nseg ? segsum[tid] : 0;
    uint64_t inc = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint64_t v = shfl_up_u64(inc, o);
      if (lane >= o) inc += v;
    }
    if (lane == 63) wave_tot[wave] = inc;
    __syncthreads();
    uint64_t wave_off = 0, total = 0;
    for (int w = 0; w < NW; ++w) {
      if (w < wave) wave_off += wave_tot[w];
      total += wave_tot[w];
    }
    if (total == 0) {  // no distribution (uniform over the block: no divergence)
      token = 0;
    } else {
      const uint64_t x = philox4x32_10(make_uint4((uint32_t)step, (uint32_t)cand[r], 0u, 0u), key).x;
      const uint64_t t = x * (total >> 32) + ((x * (total & 0xFFFFFFFFull)) >> 32);
      const uint64_t excl = wave_off + inc - mine;
      if (tid < nseg && mine > 0 && excl <= t && t < excl + mine) {
        found_seg = tid;
        found_base = excl;
      }
      __syncthreads();
      // search inside the segment (wave 0): the lane, then the entry
      if (wave == 0) {
        const int seg = found_seg;
        const int base = seg * kSegment + kPerLane * lane;
        float v[kPerLane];
        load8(base, v);
        uint64_t w[kPerLane];
        uint64_t sum = 0;
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) {
          w[e] = weight_of(v[e], m, inv_t);  // -inf past the end weighs 0
          sum += w[e];
        }
        uint64_t c = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint64_t v = shfl_up_u64(c, o);
          if (lane >= o) c += v;
        }
        const uint64_t ballot = __ballot(found_base + c > t);
        const int hit = (int)__builtin_ctzll(ballot);
        if (lane == hit) {
          uint64_t run = found_base + c - sum;
          int e = 0;
          for (; e < kPerLane - 1; ++e) {
            run += w[e];
            if (run > t) break;
          }
          red_i[0] = base + e;
        }
      }
      __syncthreads();
      token = red_i[0];
    }
  }
  if (tid == 0) {
    next_tok[r] = token;
    if (store) store[(int64_t)cand[r] * store_ld + step] = token;
    if (len) len[r] = step + 1;
    if (done && token == eos_id) done[r] = 1;
  }
}

void sample(const SampleArgs& a, hipStream_t s) {
  if (a.rows <= 0) return;
  SR_REQUIRE(a.vocab >= 1 && (a.vocab + kSegment - 1) / kSegment <= kMaxSegments, 3,
             "vocabulary too large for the sampler");
  const int greedy = a.temperature == 0.0f;
  const float inv_t = greedy ? 1.0f : (float)(1.0 / (double)a.temperature);
  const uint2 key = make_uint2((uint32_t)a.seed, (uint32_t)(a.seed >> 32));
  SR_LAUNCH(sample_kernel, dim3(a.rows), dim3(kSampleThreads), 0, s, a.logits, a.row_stride,
                     a.vocab, a.cand, a.step, inv_t, greedy, key, a.next_tok, a.done, a.len, a.store,
                     a.store_ld, a.eos_id);
  SR_CHECK_LAUNCH();
}

// ---------------------------------------------- probability as the reward
// ln p(tok) = (l_tok - m) - ln sum_i exp(l_i - m), one block per row, sums in
// a fixed order (per thread over a strided range, then the wave butterfly,
// then the waves in order).
__global__ void __launch_bounds__(256)
logprob_kernel(const float* __restrict__ logits, int64_t row_stride, int vocab, const int32_t* __restrict__ cand,
               const int32_t* __restrict__ tok, const int32_t* __restrict__ len, int step,
               float* __restrict__ lp_sum) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  if (len[r] != step + 1) return;  // uniform per block: the row was not sampled at this step
  const float* lg = logits + (int64_t)r * row_stride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float mv = -INFINITY;
  for (int i = tid; i < vocab; i += 256) mv = fmaxf(mv, lg[i]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mv = fmaxf(mv, __shfl_xor(mv, o, 64));
  if (lane == 0) red[wave] = mv;
  __syncthreads();
  const float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  for (int i = tid; i < vocab; i += 256) sum += expf(lg[i] - m);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o, 64);
  if (lane == 0) red[wave] = sum;
  __syncthreads();
  if (tid == 0) {
    const float tot = ((red[0] + red[1]) + red[2]) + red[3];
    lp_sum[cand[r]] += (lg[tok[r]] - m) - logf(tot);
  }
}

__global__ void logprob_score_kernel(const float* __restrict__ lp_sum, const int32_t* __restrict__ cand,
                                     const int32_t* __restrict__ len, int rows, float* __restrict__ score) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < rows) score[r] = len[r] > 0 ? lp_sum[cand[r]] / (float)len[r] : 0.f;
}

void logprob_accumulate(const float* logits, int64_t row_stride, int rows, int vocab, const int32_t* cand,
                        const int32_t* tok, const int32_t* len, int step, float* lp_sum, hipStream_t s) {
  if (rows <= 0) return;
  SR_LAUNCH(logprob_kernel, dim3(rows), dim3(256), 0, s, logits, row_stride, vocab, cand, tok, len, step,
                     lp_sum);
  SR_CHECK_LAUNCH();
}

void logprob_scores(const float* lp_sum, const int32_t* cand, const int32_t* len, int rows, float* score,
                    hipStream_t s) {
  if (rows <= 0) return;
  SR_LAUNCH(logprob_score_kernel, dim3((rows + 255) / 256), dim3(256), 0, s, lp_sum, cand, len, rows,
                     score);
  SR_CHECK_LAUNCH();
}

}  // namespace sr
