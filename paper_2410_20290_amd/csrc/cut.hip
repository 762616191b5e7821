// The rejection cut of section 4.2 (eqs. cutoff-threshold and accepted-set)
// and the stream compaction that packs the survivors' KV rows and state.
//
// Ranking: total order (score descending, candidate index ascending, NaN
// lowest).  A row's rank is the number of rows that precede it; the `keep`
// rows of rank < keep are accepted.  Scores are mapped to order-preserving
// unsigned keys (NaN -> 0, +0 and -0 equal), so ranks are integer-exact.
#include "common.h"
#include "kernels.h"

namespace sr {

constexpr int kCutThreads = 1024;
constexpr int kCutMax = 4096;
constexpr int kCutPer = kCutMax / kCutThreads;

__device__ __forceinline__ uint32_t order_key(float f) {
  if (f != f) return 0u;
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) == 0u) u = 0u;  // -0 == +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ bool precedes(uint32_t ka, int ca, uint32_t kb, int cb) {
  return ka > kb || (ka == kb && ca < cb);
}

// Exclusive block scan of per-thread counts (1024 threads); returns the
// exclusive prefix of this thread and writes the total to *total.
__device__ int block_excl_scan(int v, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  int off = 0, tot = 0;
  for (int w = 0; w < kCutThreads / 64; ++w) {
    if (w < wave) off += wsum[w];
    tot += wsum[w];
  }
  __syncthreads();
  *total = tot;
  return off + inc - v;
}

__device__ void rank_rows(const float* score, const int32_t* cand, int b, uint32_t* keys, int* cands,
                          int* rank) {
  for (int i = threadIdx.x; i < b; i += kCutThreads) {
    keys[i] = order_key(score[i]);
    cands[i] = cand[i];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    int rk = 0;
    if (i < b) {
      const uint32_t ki = keys[i];
      const int ci = cands[i];
      for (int j = 0; j < b; ++j) rk += precedes(keys[j], cands[j], ki, ci) ? 1 : 0;
    }
    rank[k] = rk;
  }
}

__global__ void __launch_bounds__(kCutThreads)
select_kernel(const float* __restrict__ score, const int32_t* __restrict__ cand, int b, int keep,
              int32_t* __restrict__ accept) {
  __shared__ uint32_t keys[kCutMax];
  __shared__ int cands[kCutMax];
  int rank[kCutPer];
  rank_rows(score, cand, b, keys, cands, rank);
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    if (i < b) accept[i] = rank[k] < keep ? 1 : 0;
  }
}

void select_topk(const float* score, const int32_t* cand, int b, int keep, int32_t* accept,
                 hipStream_t s) {
  SR_REQUIRE(b >= 1 && b <= kCutMax, 3, "cut supports 1..4096 rows");
  SR_LAUNCH(select_kernel, dim3(1), dim3(kCutThreads), 0, s, score, cand, b, keep, accept);
  SR_CHECK_LAUNCH();
}

__global__ void __launch_bounds__(kCutThreads) cut_kernel(CutArgs a) {
  __shared__ uint32_t keys[kCutMax];
  __shared__ int cands[kCutMax];
  __shared__ int wsum[kCutThreads / 64];
  int rank[kCutPer];
  rank_rows(a.score, a.cand, a.b, keys, cands, rank);
  int acc[kCutPer], dn[kCutPer];
  int nd = 0, nc = 0;
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    acc[k] = (i < a.b && rank[k] < a.keep) ? 1 : 0;
    dn[k] = (i < a.b && a.done[i]) ? 1 : 0;
    if (i < a.b) a.accept[i] = acc[k];
    nd += dn[k];
    nc += (acc[k] && !dn[k]) ? 1 : 0;
  }
  const int i_base = *a.i_count;
  int tot_done, tot_cont;
  int pd = block_excl_scan(nd, wsum, &tot_done);
  int pc = block_excl_scan(nc, wsum, &tot_cont);
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    if (i >= a.b) continue;
    if (dn[k]) {  // completed rows join I whether accepted or not
      const int slot = i_base + pd++;
      a.i_cand[slot] = a.cand[i];
      a.i_score[slot] = a.score[i];
      a.i_len[slot] = a.len[i];
    } else if (acc[k]) {
      const int j = pc++;
      a.src_row[j] = i;
      a.cand_out[j] = a.cand[i];
      a.len_out[j] = a.len[i];
      a.tok_out[j] = a.next_tok[i];
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    *a.i_count = i_base + tot_done;
    *a.count = tot_cont;
  }
}

void cut(const CutArgs& a, hipStream_t s) {
  SR_REQUIRE(a.b >= 1 && a.b <= kCutMax, 3, "cut supports 1..4096 rows");
  SR_LAUNCH(cut_kernel, dim3(1), dim3(kCutThreads), 0, s, a);
  SR_CHECK_LAUNCH();
}

// keep_flag -> packed source rows and count (single work-group).
__global__ void __launch_bounds__(kCutThreads)
pack_flags_kernel(const int32_t* __restrict__ flag, int b, int32_t* __restrict__ src_row,
                  int32_t* __restrict__ count) {
  __shared__ int wsum[kCutThreads / 64];
  int f[kCutPer], n = 0;
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    f[k] = (i < b && flag[i] != 0) ? 1 : 0;
    n += f[k];
  }
  int tot;
  int p = block_excl_scan(n, wsum, &tot);
#pragma unroll
  for (int k = 0; k < kCutPer; ++k) {
    const int i = threadIdx.x * kCutPer + k;
    if (f[k]) src_row[p++] = i;
  }
  if (threadIdx.x == 0) *count = tot;
}

// grid (max_rows, hkv, 2 * n_layers): copy `len` tokens of one (row, head).
__global__ void __launch_bounds__(256)
compact_kernel(const uint8_t* __restrict__ src, int64_t src_block, uint8_t* __restrict__ dst,
               int64_t dst_block, const int32_t* __restrict__ src_row, const int32_t* __restrict__ count,
               int hkv, int row_bytes, int cap_src, int cap_dst, int len) {
  const int j = blockIdx.x, h = blockIdx.y, blk = blockIdx.z;
  if (j >= *count) return;
  const int i = src_row[j];
  const uint8_t* s = src + blk * src_block + (((int64_t)i * hkv + h) * cap_src) * row_bytes;
  uint8_t* d = dst + blk * dst_block + (((int64_t)j * hkv + h) * cap_dst) * row_bytes;
  const int64_t n16 = (int64_t)len * row_bytes / 16;
  const uint4* s4 = reinterpret_cast<const uint4*>(s);
  uint4* d4 = reinterpret_cast<uint4*>(d);
  for (int64_t k = threadIdx.x; k < n16; k += 256) d4[k] = s4[k];
}

void compact(const CompactArgs& a, hipStream_t s) {
  const int32_t* src_row = a.src_row;
  const int32_t* count = a.count;
  if (a.keep_flag) {
    SR_REQUIRE(a.b >= 1 && a.b <= kCutMax, 3, "compaction supports 1..4096 rows");
    SR_LAUNCH(pack_flags_kernel, dim3(1), dim3(kCutThreads), 0, s, a.keep_flag, a.b,
                       a.scratch_src_row, a.new_count);
    SR_CHECK_LAUNCH();
    src_row = a.scratch_src_row;
    count = a.new_count;
  }
  if (a.max_rows <= 0 || a.len <= 0) return;
  const int row_bytes = a.hd * a.elem_bytes;
  SR_REQUIRE(row_bytes % 16 == 0, 3, "KV row must be a multiple of 16 bytes");
  dim3 grid(a.max_rows, a.hkv, 2 * a.n_layers);
  SR_LAUNCH(compact_kernel, grid, dim3(256), 0, s, (const uint8_t*)a.src,
                     a.src_block * a.elem_bytes, (uint8_t*)a.dst, a.dst_block * a.elem_bytes, src_row,
                     count, a.hkv, row_bytes, a.cap_src, a.cap_dst, a.len);
  SR_CHECK_LAUNCH();
}

// Best of n (score, cand) pairs; n read from the device.
__global__ void __launch_bounds__(kCutThreads)
argmax_kernel(const float* __restrict__ score, const int32_t* __restrict__ cand,
              const int32_t* __restrict__ n_dev, int n_max, int32_t* __restrict__ best) {
  __shared__ uint32_t sk[kCutThreads / 64];
  __shared__ int sc[kCutThreads / 64], si[kCutThreads / 64];
  const int n = min(*n_dev, n_max);
  uint32_t bk = 0;
  int bc = 0x7FFFFFFF, bi = -1;
  for (int i = threadIdx.x; i < n; i += kCutThreads) {
    const uint32_t k = order_key(score[i]);
    const int c = cand[i];
    if (bi < 0 || precedes(k, c, bk, bc)) { bk = k; bc = c; bi = i; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t ok = __shfl_xor(bk, o, 64);
    const int oc = __shfl_xor(bc, o, 64), oi = __shfl_xor(bi, o, 64);
    if (oi >= 0 && (bi < 0 || precedes(ok, oc, bk, bc))) { bk = ok; bc = oc; bi = oi; }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) { sk[wave] = bk; sc[wave] = bc; si[wave] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 0; w < kCutThreads / 64; ++w)
      if (si[w] >= 0 && (bi < 0 || precedes(sk[w], sc[w], bk, bc))) { bk = sk[w]; bc = sc[w]; bi = si[w]; }
    best[0] = bi;
  }
}

void argmax_best(const float* score, const int32_t* cand, const int32_t* n_dev, int n_max,
                 int32_t* best, hipStream_t s) {
  SR_LAUNCH(argmax_kernel, dim3(1), dim3(kCutThreads), 0, s, score, cand, n_dev, n_max, best);
  SR_CHECK_LAUNCH();
}

}  // namespace sr
