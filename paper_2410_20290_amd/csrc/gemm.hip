// Projections of the decoder (QKV, O, gate|up + SwiGLU, down, LM head):
// C[m][n] = sum_k A[m][k] * B[n][k], A = activations [M][lda], B = weights
// [N][ldb] (both K-contiguous), fp32 accumulation, fused epilogues.
//
// bf16: MFMA tiles staged through LDS (by LDS DMA for the main kernels):
// 256 x 256 and 256 x 128 tiles of v_mfma_f32_32x32x16_bf16 for hundreds of
// rows and more, streaming tiles of v_mfma_f32_16x16x32_bf16 for up to 128
// rows.  fp32: a plain LDS-tiled FMA kernel (used by the fp32 model).
// Split-K writes fp32 partials [split][M][Nout] that a consumer sums in
// split order, so results do not depend on scheduling.
#include <cstdlib>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace sr {

// ---------------------------------------------------------------- epilogues
struct EpiArgs {
  int mode;       // GemmEpi
  void* out;      // destination (type per mode)
  int ldo;        // leading dimension of out (elements)
  int out_bf16;   // for EPI_STORE and EPI_SWIGLU: 1 = bf16 out, 0 = fp32 out
};

__device__ __forceinline__ float silu(float x) { return x / (1.0f + __expf(-x)); }

__device__ __forceinline__ void store_out(const EpiArgs& e, int m, int n, float v) {
  if (e.out_bf16)
    reinterpret_cast<bf16_t*>(e.out)[(int64_t)m * e.ldo + n] = f32_to_bf16(v);
  else
    reinterpret_cast<float*>(e.out)[(int64_t)m * e.ldo + n] = v;
}

// Single-output epilogue (modes EPI_STORE, EPI_RESID).
__device__ __forceinline__ void epi_one(const EpiArgs& e, int m, int n, float v) {
  if (e.mode == EPI_RESID) {
    float* h = reinterpret_cast<float*>(e.out) + (int64_t)m * e.ldo + n;
    *h = *h + v;
  } else {
    store_out(e, m, n, v);
  }
}

// ------------------------------------------------------------ tile order
// Work-groups are dealt round-robin to the 8 XCDs, each with its own L2.  A
// 1-D grid of 8 * C groups is remapped so that XCD x runs the consecutive
// logical tiles [x C, (x + 1) C); logical tiles are ordered split-major, then
// in groups of up to 8 row tiles with the row tile fastest, so tiles that
// share a weight panel (same column tile and split) run on one XCD at about
// the same time, and tiles that share an activation panel stay close.
struct TileIdx {
  int m, n, split;
  bool valid;
};

__device__ __forceinline__ TileIdx tile_of(int nm, int nn, int splits) {
  const int total = nm * nn * splits;
  const int per_xcd = (total + 7) / 8;
  const int g = blockIdx.x;
  const int pid = (g % 8) * per_xcd + g / 8;
  TileIdx t;
  t.valid = pid < total;
  const int per_split = nm * nn;
  t.split = pid / per_split;
  const int q = pid % per_split;
  const int gm = min(nm, 8);
  const int in_group = gm * nn;
  const int grp = q / in_group;
  const int first_m = grp * gm;
  const int size_m = min(nm - first_m, gm);
  const int r = q % in_group;
  t.m = first_m + r % size_m;
  t.n = r / size_m;
  return t;
}

static inline dim3 tile_grid(int nm, int nn, int splits) {
  const int total = nm * nn * splits;
  return dim3(8 * ((total + 7) / 8));
}

// ------------------------------------------------------------ tile epilogue
// The 32x32x16 kernels below multiply with the weight fragment as the first
// MFMA operand, so each wave accumulates the transpose of its output tile:
// element e of lane l of acc[i][j] is tile row 32 i + l % 32, tile column
// 32 j + 8 (e / 4) + 4 (l / 32) + e % 4, i.e. runs of four consecutive
// columns.  A wave writes its tile as 16-byte chunks (four floats) into its
// own 32 KB of the then idle LDS, 8192 / CL rows per pass (CL floats per
// row, chunk c of row r in slot c ^ key(r)), and reads it back along rows,
// so that global stores (and residual reads) are contiguous row runs of 16
// (fp32) or 8 (bf16) bytes per lane rather than scattered single elements.
//
// Paired tiles: acc[i][2 jj] holds the gate and acc[i][2 jj + 1] the up
// projection of output columns 32 jj + ...; without partials the SwiGLU
// product is staged (MERGE, CL = 16 TJ); with partials gate and up are
// staged side by side (CL = 32 TJ) and go to columns n and N + n of the
// [split][M][2N] partial rows.
template <int CL>
__device__ __forceinline__ int stage_slot(int r, int c) {
  constexpr int CPR = CL / 4, RB = CL * 4;  // chunks and bytes per row
  const int key = RB >= 256 ? r % CPR : (r / (256 / RB)) % CPR;
  return r * CL + 4 * (c ^ key);
}

__device__ __forceinline__ void store4(float* dst, f32x4 v) { *reinterpret_cast<f32x4*>(dst) = v; }

__device__ __forceinline__ void store4(bf16_t* dst, f32x4 v) {
  const uint32_t lo = f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  const uint32_t hi = f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  *reinterpret_cast<uint2*>(dst) = uint2{lo, hi};
}

// row0, col0: output row and output column of the wave tile's first row and
// column (for paired tiles the SwiGLU / partial column, not the weight row).
// Wave tiles wholly inside the output with 16-byte aligned rows take the
// unrolled path (residual rows of a pass loaded before its staging); edge
// tiles store element by element.
template <int TI, int TJ, bool PAIRED, bool MERGE>
__device__ __forceinline__ void tile_epilogue_32(const f32x16 (&acc)[TI][TJ], float* st, int lane, int row0,
                                                 int col0, int M, int N, int split, const EpiArgs& epi,
                                                 float* __restrict__ partial) {
  static_assert(!MERGE || PAIRED, "only paired tiles merge gate and up");
  constexpr int CL = MERGE ? 16 * TJ : 32 * TJ;                 // staged floats per row
  constexpr int LPR = CL / 4;                                   // lanes per row on read-back
  constexpr int RPI = 64 / LPR;                                 // rows per read-back instruction
  constexpr int RP = 8192 / CL < 32 * TI ? 8192 / CL : 32 * TI;  // rows per pass
  constexpr int NP = 32 * TI / RP, NQ = RP / RPI;
  constexpr int WCOLS = PAIRED ? 16 * TJ : 32 * TJ;             // output columns of the wave tile
  static_assert(LPR <= 64 && RP % 32 == 0 && RP % RPI == 0, "epilogue shape");
  const int lr = lane & 31, lh = lane >> 5;
  const int rr = lane / LPR, cc = 4 * (lane % LPR);  // read-back row within a group, staged column

  // staged column cc -> output column n (and the gate or up half of a
  // paired partial row)
  int n = col0 + cc;
  bool up = false;
  if (PAIRED && !MERGE) {
    const int j = cc / 32;
    n = col0 + 32 * (j / 2) + cc % 32;
    up = j & 1;
  }
  const bool to_part = partial != nullptr;
  const bool resid = !PAIRED && !to_part && epi.mode == EPI_RESID;
  const bool bf = !to_part && !resid && epi.out_bf16;
  const int64_t ld = to_part ? (PAIRED ? 2 * (int64_t)N : (int64_t)N) : (int64_t)epi.ldo;
  const bool aligned = to_part ? (N % 4 == 0 && (reinterpret_cast<uintptr_t>(partial) & 15) == 0)
                               : (epi.ldo % 4 == 0 && (reinterpret_cast<uintptr_t>(epi.out) & 15) == 0);
  const bool interior = aligned && row0 + 32 * TI <= M && col0 + WCOLS <= N;
  const int64_t col = n + (up ? N : 0);
  float* const fbase = to_part ? partial + (int64_t)split * M * ld : reinterpret_cast<float*>(epi.out);
  bf16_t* const bbase = reinterpret_cast<bf16_t*>(epi.out);

#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int prow = row0 + p * RP;
    f32x4 old[NQ];
    if (interior && resid) {
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        old[q] = *reinterpret_cast<const f32x4*>(fbase + (int64_t)(prow + q * RPI + rr) * ld + col);
    }
#pragma unroll
    for (int ii = 0; ii < RP / 32; ++ii) {
      const int i = p * (RP / 32) + ii;
      const int r = ii * 32 + lr;
#pragma unroll
      for (int j = 0; j < (MERGE ? TJ / 2 : TJ); ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          f32x4 v;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if constexpr (MERGE) v[k] = silu(acc[i][2 * j][4 * g + k]) * acc[i][2 * j + 1][4 * g + k];
            else v[k] = acc[i][j][4 * g + k];
          }
          *reinterpret_cast<f32x4*>(st + stage_slot<CL>(r, 8 * j + 2 * g + lh)) = v;
        }
    }
    if (interior) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int r = q * RPI + rr;
        f32x4 v = *reinterpret_cast<const f32x4*>(st + stage_slot<CL>(r, cc / 4));
        const int64_t off = (int64_t)(prow + r) * ld + col;
        if (resid) v += old[q];
        if (bf) store4(bbase + off, v);
        else store4(fbase + off, v);
      }
    } else {
#pragma unroll 1
      for (int q = 0; q < NQ; ++q) {
        const int r = q * RPI + rr;
        const f32x4 v = *reinterpret_cast<const f32x4*>(st + stage_slot<CL>(r, cc / 4));
        const int m = prow + r;
        if (m >= M) continue;
        const int64_t off = (int64_t)m * ld + col;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (n + k >= N) break;
          if (resid) fbase[off + k] += v[k];
          else if (bf) bbase[off + k] = f32_to_bf16(v[k]);
          else fbase[off + k] = v[k];
        }
      }
    }
  }
}

// ------------------------------------------------------------ bf16 MFMA GEMM
// Block tile BM x BN (x2 when PAIRED: gate rows n and up rows pair_off + n),
// K step BK, wave tile WM x WN.  PAIRED epilogue: silu(gate) * up.
template <int BM, int BN, int BK, int WM, int WN, bool PAIRED>
__global__ void __launch_bounds__((BM / WM) * (BN / WN) * 64)
gemm_bf16_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb,
                 int64_t pair_off, int M, int N, int K, int k_per_split, EpiArgs epi,
                 float* __restrict__ partial) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  constexpr int NB = PAIRED ? 2 : 1;
  constexpr int PAD = 8;
  constexpr int LDS_ROW = BK + PAD;  // bf16 elements per LDS row
  constexpr int TM = WM / 16, TN = WN / 16;
  constexpr int CH_ROW = BK / 8;     // 16-byte chunks per row
  constexpr int A_CH = BM * CH_ROW, B_CH = NB * BN * CH_ROW;
  constexpr int A_IT = (A_CH + NT - 1) / NT, B_IT = (B_CH + NT - 1) / NT;

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][NB * BN * LDS_ROW];

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN - 1) / BN, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / (BN / WN)) * WM, wn0 = (wave % (BN / WN)) * WN;
  const int m0 = tile.m * BM, n0 = tile.n * BN;
  const int k_begin = tile.split * k_per_split;
  const int k_end = min(K, k_begin + k_per_split);
  const int nk = (k_end - k_begin) / BK;

  f32x4 acc[NB][TM][TN];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[b][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  uint4 ra[A_IT], rb[B_IT];
  // unconditional loads (rows clamped, out-of-range rows zeroed by a select)
  auto load_global = [&](int kt) {
    const int kb = k_begin + kt * BK;
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
      const int c = min(tid + it * NT, A_CH - 1);
      const int r = c / CH_ROW, cc = c % CH_ROW;
      const int m = m0 + r;
      const uint4 v = *reinterpret_cast<const uint4*>(A + (int64_t)min(m, M - 1) * lda + kb + cc * 8);
      ra[it] = m < M ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      const int c = min(tid + it * NT, B_CH - 1);
      const int r = c / CH_ROW, cc = c % CH_ROW;
      const int blk = r / BN, rr = r % BN;
      const int n = n0 + rr;
      const uint4 v =
          *reinterpret_cast<const uint4*>(B + blk * pair_off + (int64_t)min(n, N - 1) * ldb + kb + cc * 8);
      rb[it] = n < N ? v : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
      int c = tid + it * NT;
      if (c < A_CH) {
        int r = c / CH_ROW, cc = c % CH_ROW;
        *reinterpret_cast<uint4*>(&As[buf][r * LDS_ROW + cc * 8]) = ra[it];
      }
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      int c = tid + it * NT;
      if (c < B_CH) {
        int r = c / CH_ROW, cc = c % CH_ROW;
        *reinterpret_cast<uint4*>(&Bs[buf][r * LDS_ROW + cc * 8]) = rb[it];
      }
    }
  };

  if (nk > 0) {
    load_global(0);
    store_lds(0);
  }
  __syncthreads();
  const int fr = lane & 15, fg = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      bf16x8 af[TM];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&As[buf][(wm0 + i * 16 + fr) * LDS_ROW + ks + fg * 8]);
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          bf16x8 bfr = *reinterpret_cast<const bf16x8*>(
              &Bs[buf][(b * BN + wn0 + j * 16 + fr) * LDS_ROW + ks + fg * 8]);
#pragma unroll
          for (int i = 0; i < TM; ++i)
            acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr, acc[b][i][j], 0, 0, 0);
        }
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  // Accumulator layout: lane holds rows 4*(lane/16) + e, column lane % 16.
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        int m = m0 + wm0 + i * 16 + fg * 4 + e;
        int n = n0 + wn0 + j * 16 + fr;
        if (m >= M || n >= N) continue;
        if (partial) {
          const int nout = NB * N;
          float* p = partial + ((int64_t)tile.split * M + m) * nout;
          p[n] = acc[0][i][j][e];
          if (PAIRED) p[N + n] = acc[NB - 1][i][j][e];
        } else if (PAIRED) {
          store_out(epi, m, n, silu(acc[0][i][j][e]) * acc[NB - 1][i][j][e]);
        } else {
          epi_one(epi, m, n, acc[0][i][j][e]);
        }
      }
}


// ------------------------------------------------- bf16 MFMA GEMM, large M
// 256 x 256 block tile (PAIRED: 128 output columns, gate and up rows
// interleaved in groups of 32 so one wave holds both for its columns),
// K step 64, 4 waves each owning a 128 x 128 tile of 4 x 4
// v_mfma_f32_32x32x16_bf16 accumulators (256 fp32 per lane).  The next K
// tile is fetched into registers while the current one is multiplied from
// LDS; ~2k MFMA cycles per wave per iteration cover the fetch latency.
template <bool PAIRED>
__global__ void __launch_bounds__(256)
gemm_big_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb,
                int64_t pair_off, int M, int N, int K, int k_per_split, EpiArgs epi,
                float* __restrict__ partial) {
  constexpr int BM = 256, BNL = 256, BK = 64, PAD = 8, LDS_ROW = BK + PAD;
  constexpr int BN_OUT = PAIRED ? 128 : 256;   // output columns per block
  constexpr int CH_ROW = BK / 8;               // 8 chunks of 16 B per row
  constexpr int IT = BM * CH_ROW / 256;        // 8 chunks per thread (A and B alike)
  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BNL * LDS_ROW];

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN_OUT - 1) / BN_OUT, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 128, wn0 = (wave & 1) * 128;
  const int m0 = tile.m * BM, n0 = tile.n * BN_OUT;
  const int k_begin = tile.split * k_per_split;
  const int k_end = min(K, k_begin + k_per_split);
  const int nk = (k_end - k_begin) / BK;

  // B row of LDS row r
  auto brow = [&](int r, int64_t* off, int* n) {
    if (PAIRED) {
      const int grp = r >> 5, blk = grp & 1;
      *n = n0 + (grp >> 1) * 32 + (r & 31);
      *off = blk * pair_off;
    } else {
      *n = n0 + r;
      *off = 0;
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  uint4 ra[IT], rb[IT];
  auto load_global = [&](int kt) {
    const int kb = k_begin + kt * BK;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int c = tid + it * 256;
      const int r = c / CH_ROW, cc = c % CH_ROW;
      const int m = m0 + r;
      const uint4 va = *reinterpret_cast<const uint4*>(A + (int64_t)min(m, M - 1) * lda + kb + cc * 8);
      ra[it] = m < M ? va : make_uint4(0, 0, 0, 0);
      int64_t off;
      int n;
      brow(r, &off, &n);
      const uint4 vb = *reinterpret_cast<const uint4*>(B + off + (int64_t)min(n, N - 1) * ldb + kb + cc * 8);
      rb[it] = n < N ? vb : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int c = tid + it * 256;
      const int r = c / CH_ROW, cc = c % CH_ROW;
      *reinterpret_cast<uint4*>(&As[buf][r * LDS_ROW + cc * 8]) = ra[it];
      *reinterpret_cast<uint4*>(&Bs[buf][r * LDS_ROW + cc * 8]) = rb[it];
    }
  };

  if (nk > 0) {
    load_global(0);
    store_lds(0);
  }
  __syncthreads();
  const int fr = lane & 31, fg = lane >> 5;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_global(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&As[buf][(wm0 + i * 32 + fr) * LDS_ROW + ks + fg * 8]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(&Bs[buf][(wn0 + j * 32 + fr) * LDS_ROW + ks + fg * 8]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_lds(buf ^ 1);
    __syncthreads();
  }

  // 32x32 accumulator layout: element e of lane l is row 8*(e/4) + 4*(l/32) + e%4, column l%32.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int m = m0 + wm0 + i * 32 + 8 * (e >> 2) + 4 * fg + (e & 3);
      if (m >= M) continue;
      if (PAIRED) {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int n = n0 + (wn0 >> 1) + jj * 32 + fr;
          if (n >= N) continue;
          const float g = acc[i][2 * jj][e], u = acc[i][2 * jj + 1][e];
          if (partial) {
            float* p = partial + ((int64_t)tile.split * M + m) * (2 * (int64_t)N);
            p[n] = g;
            p[N + n] = u;
          } else {
            store_out(epi, m, n, silu(g) * u);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + wn0 + j * 32 + fr;
          if (n >= N) continue;
          if (partial)
            partial[((int64_t)tile.split * M + m) * N + n] = acc[i][j][e];
          else
            epi_one(epi, m, n, acc[i][j][e]);
        }
      }
    }
}


// ------------------------------------- bf16 MFMA GEMM, LDS-DMA pipeline
// 256 x 256 block tile (PAIRED: gate and up rows interleaved in groups of 32,
// 128 output columns), K step 64, two LDS stages of 64 KB.  Operand tiles go
// from memory straight into LDS with buffer loads (buffer_load_dwordx4 ...
// lds: no staging registers, the K step as the scalar offset, 1-4 % faster
// than global_load_lds_dwordx4 with 64-bit lane addresses); each
// instruction moves 8 rows of 128 bytes, so every request to L2 is a whole
// 128-byte line.  A K step is four quarter steps of 16
// MFMAs per wave (4 waves, each a 128 x 128 tile of 4 x 4
// v_mfma_f32_32x32x16_bf16 accumulators).  The fragments of quarters 1-3
// are read under the MFMAs of quarters 0 and 1 (three register sets that
// rotate from step to step), so the buffer is free after quarter 1: the
// DMAs of the step after next are spread over quarters 2 and 3 (A rows, then
// B rows), which keeps the vector-memory path from backing up into the MFMA
// issue.  One barrier per step, after quarter 1: the buffer has been read by
// all waves and the next step (whose DMAs went out under quarters 2 and 3 of
// the step before) has landed in all of them.  LDS rows hold eight
// 16-byte chunks; chunk c of tile row r sits in slot c ^ (r & 7) ^ ((r >> 3) & 3)
// (a function of r mod 32, so fragment blocks of 32 rows share it), which puts the fragment reads of any 8 or 16 consecutive rows on distinct
// banks.
#define SR_VM_BARRIER(n) asm volatile("s_waitcnt vmcnt(" #n ") lgkmcnt(0)\n\ts_barrier" ::: "memory")

//
// BRING = 3 (a few hundred rows, where every weight tile comes from HBM and
// is shared by few row tiles): the weight rows get a ring of three buffers
// of their own, filled three steps ahead, while the activation rows (in L2)
// keep two; 160 KB of LDS.
template <bool PAIRED, int BRING>
__global__ void __launch_bounds__(256)
gemm_dma_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb,
                int64_t pair_off, int M, int N, int K, int k_per_split, EpiArgs epi,
                float* __restrict__ partial) {
  constexpr int BM = 256, BNL = 256, BK = 64;
  constexpr int BN_OUT = PAIRED ? 128 : 256;
  constexpr int STAGE = (BM + BNL) * BK;  // bf16 elements per stage
  constexpr int HALF = BM * BK;           // bf16 elements of the A (or B) rows of a stage
  static_assert(BRING == 2 || BRING == 3, "weight ring depth");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[BRING == 2 ? 2 * STAGE : 2 * HALF + 3 * HALF];
  // A rows of ring slot `a`, B rows of ring slot `b`
  auto a_base = [&](int a) { return lds + (BRING == 2 ? a * STAGE : a * HALF); };
  auto b_base = [&](int b) { return lds + (BRING == 2 ? b * STAGE + HALF : 2 * HALF + b * HALF); };

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN_OUT - 1) / BN_OUT, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave >> 1) * 128, wn0 = (wave & 1) * 128;
  const int m0 = tile.m * BM, n0 = tile.n * BN_OUT;
  const int k_begin = tile.split * k_per_split;
  const int nk = k_per_split / BK;

  // DMA sources: A and B each fill a stage with 32 wave instructions of 1 KB
  // (8 rows of 128 bytes); wave w issues rows 8 (w + 4 i) .. + 7, i < 8.
  // Lane l writes slot l % 8 of row l / 8, so it fetches the chunk stored
  // there.  Rows past M or N are clamped (their results are never stored).
  uint32_t aoff[8], boff[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = 8 * (wave + 4 * i) + (lane >> 3);
    const int c = (lane & 7) ^ (r & 7) ^ ((r >> 3) & 3);
    aoff[i] = (uint32_t)(((int64_t)min(m0 + r, M - 1) * lda + c * 8) * 2);
    int n;
    int64_t off = 0;
    if (PAIRED) {
      const int grp = r >> 5;
      n = n0 + (grp >> 1) * 32 + (r & 31);
      off = (grp & 1) * pair_off;
    } else {
      n = n0 + r;
    }
    boff[i] = (uint32_t)((off + (int64_t)min(n, N - 1) * ldb + c * 8) * 2);
  }
  const BufRsrc ra = buf_rsrc(A + k_begin), rb = buf_rsrc(B + k_begin);
  // half h of stage `st` into ring slot `buf`: the A rows (h = 0) or the B
  // rows (h = 1), 8 instructions per wave
  auto issue_half = [&](int st, int buf, int h) {
    bf16_t* dst = h ? b_base(buf) : a_base(buf);
#pragma unroll
    for (int i = 0; i < 8; ++i) dma16(h ? rb : ra, h ? boff[i] : aoff[i], st * BK * 2, dst + (wave + 4 * i) * 512);
  };

  // Fragment reads: lane l holds row l % 32 of a 32-row block, K chunk
  // 2 q + l / 32 of quarter q.
  const int fr = lane & 31, fg = lane >> 5;
  const int sw = (fr & 7) ^ ((fr >> 3) & 3);
  int foff[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) foff[q] = fr * BK + 8 * ((2 * q + fg) ^ sw);
  auto read_frags = [&](int abuf, int bbuf, int q, bf16x8(&af)[4], bf16x8(&bfr)[4]) {
    const bf16_t* sa = a_base(abuf) + foff[q];
    const bf16_t* sb = b_base(bbuf) + foff[q];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sa + (wm0 + 32 * i) * BK);
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(sb + (wn0 + 32 * j) * BK);
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  auto mfma = [&](const bf16x8(&af)[4], const bf16x8(&bfr)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
  };
  // instruction interleavings before the step barrier: (MFMA, fragment
  // read) x 16; (MFMA, read) x 8 then 8 MFMAs (after it the order is written
  // out: the scheduler bunched the copies behind one MFMA)
  auto reads16 = [] {
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto reads8 = [] {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // Every step issues the DMAs of the step after next; past the last step
  // the source is clamped to the last step (data never read), which keeps
  // every wait below the same at each step.
  issue_half(0, 0, 0);
  issue_half(0, 0, 1);
  issue_half(min(1, nk - 1), 1, 0);
  issue_half(min(1, nk - 1), 1, 1);
  if constexpr (BRING == 3) {
    issue_half(min(2, nk - 1), 2, 1);
    SR_VM_BARRIER(24);
  } else {
    SR_VM_BARRIER(16);
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): no scalar loads in flight past here
  bf16x8 a0[4], b0[4], a1[4], b1[4], a2[4], b2[4];
  read_frags(0, 0, 0, a0, b0);
  // One K step with its quarter 0 in (xa, xb); quarter 3 reuses those
  // registers and the next step's quarter 0 goes to (ya, yb).  bb, bbn: B
  // ring slots of steps t and t + 1.  One barrier per step, after quarter 1:
  // every wave has read the buffers of step t, and step t + 1 has landed
  // (all but this wave's newest DMAs: none with two stages, the B rows of
  // step t + 2 with three).  Then the A rows of step t + 2 go out under
  // quarter 2 and the B rows of step t + BRING under quarter 3.
  auto step = [&](int t, int bb, int bbn, bf16x8(&xa)[4], bf16x8(&xb)[4], bf16x8(&ya)[4], bf16x8(&yb)[4],
                  bf16x8(&za)[4], bf16x8(&zb)[4]) {
    const int buf = t & 1;
    const int nx = min(t + 2, nk - 1), nxb = min(t + BRING, nk - 1);
    read_frags(buf, bb, 1, ya, yb);
    read_frags(buf, bb, 2, za, zb);
    mfma(xa, xb);
    reads16();
    read_frags(buf, bb, 3, xa, xb);
    mfma(ya, yb);
    reads8();
    if constexpr (BRING == 3) SR_VM_BARRIER(8);
    else SR_VM_BARRIER(0);
    __builtin_amdgcn_sched_barrier(0);
    // Quarter 2 with the A rows of step t + 2 and the next step's quarter-0
    // fragments (after the last step a stale buffer that is never used):
    // one copy and one read per pair of MFMAs, in this order.
    {
      bf16_t* dst = a_base(buf);
      const bf16_t* sa = a_base(buf ^ 1) + foff[0];
      const bf16_t* sb = b_base(bbn) + foff[0];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const int i = p >> 1, j = (p & 1) * 2;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(zb[j], za[i], acc[i][j], 0, 0, 0);
        acc[i][j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(zb[j + 1], za[i], acc[i][j + 1], 0, 0, 0);
        dma16(ra, aoff[p], nx * BK * 2, dst + (wave + 4 * p) * 512);
        if (p < 4) ya[p] = *reinterpret_cast<const bf16x8*>(sa + (wm0 + 32 * p) * BK);
        else yb[p - 4] = *reinterpret_cast<const bf16x8*>(sb + (wn0 + 32 * (p - 4)) * BK);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // Quarter 3 with the B rows of step t + BRING, one copy per MFMA pair.
    {
      bf16_t* dst = b_base(bb);
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const int i = p >> 1, j = (p & 1) * 2;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xb[j], xa[i], acc[i][j], 0, 0, 0);
        acc[i][j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xb[j + 1], xa[i], acc[i][j + 1], 0, 0, 0);
        dma16(rb, boff[p], nxb * BK * 2, dst + (wave + 4 * p) * 512);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  for (int t = 0; t < nk; t += 3) {
    // B ring slots: t % 3 with three (t is a multiple of 3 here), t % 2 with two
    const int s0 = BRING == 3 ? 0 : (t & 1), s1 = BRING == 3 ? 1 : s0 ^ 1, s2 = BRING == 3 ? 2 : s0;
    step(t, s0, s1, a0, b0, a1, b1, a2, b2);
    if (t + 1 < nk) step(t + 1, s1, s2, a1, b1, a2, b2, a0, b0);
    if (t + 2 < nk) step(t + 2, s2, BRING == 3 ? 0 : s1, a2, b2, a0, b0, a1, b1);
  }
  // no DMA may still be writing LDS and no wave still reading it
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  float* st = reinterpret_cast<float*>(lds) + wave * 8192;
  if (PAIRED && !partial)
    tile_epilogue_32<4, 4, PAIRED, PAIRED>(acc, st, lane, m0 + wm0, n0 + wn0 / 2, M, N, tile.split, epi, partial);
  else
    tile_epilogue_32<4, 4, PAIRED, false>(acc, st, lane, m0 + wm0, n0 + (PAIRED ? wn0 / 2 : wn0), M, N, tile.split,
                                          epi, partial);
}
#undef SR_VM_BARRIER


// ------------------------- bf16 MFMA GEMM, a few hundred rows (LDS DMA)
// 256 x 128 block tile (PAIRED: gate and up rows interleaved in groups of
// 32, 64 output columns), K step 64, three LDS stages of 48 KB.  With a
// third stage the buffer refilled during step t (that of step t - 1) is
// free from its start, so the 12 DMA instructions per wave of the step after
// next are spread over quarter steps 0-2 and the data of step t + 1 has a
// whole step to land; one barrier per step, before quarter 3.  4 waves, each
// a 128 x 64 tile of 4 x 2 v_mfma_f32_32x32x16_bf16 accumulators; LDS rows,
// their swizzle and the buffer-load copies as in the 256 x 256 kernel.
#define SR_VMB3(n) asm volatile("s_waitcnt vmcnt(" #n ") lgkmcnt(0)\n\ts_barrier" ::: "memory")

template <bool PAIRED>
__global__ void __launch_bounds__(256)
gemm_dma3_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb,
                 int64_t pair_off, int M, int N, int K, int k_per_split, EpiArgs epi,
                 float* __restrict__ partial) {
  constexpr int BM = 256, BNL = 128, BK = 64, NST = 3;
  constexpr int BN_OUT = PAIRED ? 64 : 128;
  constexpr int STAGE = (BM + BNL) * BK;      // bf16 elements per stage
  constexpr int DA = BM / 32, DB = BNL / 32;  // DMA instructions per wave per stage
  static_assert(DA + DB == 12, "the wait count below assumes 12 DMAs per wave per stage");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NST * STAGE];

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN_OUT - 1) / BN_OUT, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave >> 1) * 128, wn0 = (wave & 1) * 64;
  const int m0 = tile.m * BM, n0 = tile.n * BN_OUT;
  const int k_begin = tile.split * k_per_split;
  const int nk = k_per_split / BK;

  // DMA sources: instruction i of a wave moves tile rows 8 (w + 4 i) .. + 7
  // (A rows for i < DA, then B rows); lane l writes slot l % 8 of row l / 8.
  uint32_t aoff[DA], boff[DB];
#pragma unroll
  for (int i = 0; i < DA; ++i) {
    const int r = 8 * (wave + 4 * i) + (lane >> 3);
    const int c = (lane & 7) ^ (r & 7) ^ ((r >> 3) & 3);
    aoff[i] = (uint32_t)(((int64_t)min(m0 + r, M - 1) * lda + c * 8) * 2);
  }
#pragma unroll
  for (int i = 0; i < DB; ++i) {
    const int r = 8 * (wave + 4 * i) + (lane >> 3);
    const int c = (lane & 7) ^ (r & 7) ^ ((r >> 3) & 3);
    int n;
    int64_t off = 0;
    if (PAIRED) {
      const int grp = r >> 5;
      n = n0 + (grp >> 1) * 32 + (r & 31);
      off = (grp & 1) * pair_off;
    } else {
      n = n0 + r;
    }
    boff[i] = (uint32_t)((off + (int64_t)min(n, N - 1) * ldb + c * 8) * 2);
  }
  const BufRsrc ra = buf_rsrc(A + k_begin), rb = buf_rsrc(B + k_begin);
  auto dma = [&](int st, int buf, int i) {
    bf16_t* sa = lds + buf * STAGE;
    const int kb = st * BK * 2;
    if (i < DA) dma16(ra, aoff[i], kb, sa + (wave + 4 * i) * 512);
    else dma16(rb, boff[i - DA], kb, sa + BM * BK + (wave + 4 * (i - DA)) * 512);
  };

  const int fr = lane & 31, fg = lane >> 5;
  const int sw = (fr & 7) ^ ((fr >> 3) & 3);
  int foff[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) foff[q] = fr * BK + 8 * ((2 * q + fg) ^ sw);
  auto read_frags = [&](int buf, int q, bf16x8(&af)[4], bf16x8(&bfr)[2]) {
    const bf16_t* sa = lds + buf * STAGE + foff[q];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(sa + (wm0 + 32 * i) * BK);
#pragma unroll
    for (int j = 0; j < 2; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(sa + (BM + wn0 + 32 * j) * BK);
  };
  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  // Every step issues the DMAs of the step after next (clamped to the last
  // step past the end: data never read), so every wait is the same.
#pragma unroll
  for (int i = 0; i < DA + DB; ++i) dma(0, 0, i);
#pragma unroll
  for (int i = 0; i < DA + DB; ++i) dma(min(1, nk - 1), 1, i);
  SR_VMB3(12);  // step 0 landed
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): no scalar loads in flight past here
  bf16x8 a0[4], b0[2], a1[4], b1[2];
  read_frags(0, 0, a0, b0);
  // One step; `live`: the step after next exists and is fetched (the last
  // two steps fetch nothing and wait for every copy, so no copy is in flight
  // at the end).
  // One quarter step: the MFMAs of (af, bfr), the fragments of quarter rq
  // of buffer rbuf into (na, nb2) and, with FETCH, copies d0 .. d0 + 3 of
  // step nx into buffer wb, in the order (MFMA, read, MFMA, copy) x 4 and
  // the two B reads (written out: the scheduler bunched the copies).
  auto quarter = [&](auto fetch, const bf16x8(&af)[4], const bf16x8(&bfr)[2], int rbuf, int rq, bf16x8(&na)[4],
                     bf16x8(&nb2)[2], int nx, int wb, int d0) {
    constexpr bool FETCH = decltype(fetch)::value;
    const bf16_t* sa = lds + rbuf * STAGE + foff[rq];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[0], af[i], acc[i][0], 0, 0, 0);
      na[i] = *reinterpret_cast<const bf16x8*>(sa + (wm0 + 32 * i) * BK);
      acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[1], af[i], acc[i][1], 0, 0, 0);
      if constexpr (FETCH) dma(nx, wb, d0 + i);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) nb2[j] = *reinterpret_cast<const bf16x8*>(sa + (BM + wn0 + 32 * j) * BK);
    __builtin_amdgcn_sched_barrier(0);
  };
  auto step = [&](auto live, int t) {
    constexpr bool FETCH = decltype(live)::value;
    const int buf = t % 3, nb = (t + 1) % 3, wb = (t + 2) % 3;
    const int nx = t + 2;
    quarter(live, a0, b0, buf, 1, a1, b1, nx, wb, 0);
    quarter(live, a1, b1, buf, 2, a0, b0, nx, wb, 4);
    quarter(live, a0, b0, buf, 3, a1, b1, nx, wb, 8);
    // step t + 1 landed (all but this wave's 12 newest DMAs; none in the
    // last two steps) in every wave, and every wave has read all it needs
    // of buffer `buf`
    if constexpr (FETCH) SR_VMB3(12);
    else SR_VMB3(0);
    __builtin_amdgcn_sched_barrier(0);
    // (after the last step this reads a stale buffer that is never used)
    quarter(std::false_type{}, a1, b1, nb, 0, a0, b0, 0, 0, 0);
  };
  int t = 0;
  for (; t < nk - 2; ++t) step(std::true_type{}, t);
  for (; t < nk; ++t) step(std::false_type{}, t);
  // no DMA may still be writing LDS and no wave still reading it
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  float* st = reinterpret_cast<float*>(lds) + wave * 8192;
  if (PAIRED && !partial)
    tile_epilogue_32<4, 2, PAIRED, PAIRED>(acc, st, lane, m0 + wm0, n0 + wn0 / 2, M, N, tile.split, epi, partial);
  else
    tile_epilogue_32<4, 2, PAIRED, false>(acc, st, lane, m0 + wm0, n0 + (PAIRED ? wn0 / 2 : wn0), M, N, tile.split,
                                          epi, partial);
}
#undef SR_VMB3

// s_waitcnt vmcnt(N) lgkmcnt(0) then s_barrier, N a compile-time count; and
// the same with N = A * D for a run-time a <= A (copies of a later stages of
// D instructions each may stay in flight).
template <int N>
__device__ __forceinline__ void vm_barrier() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
#define SR_VMB_CASE(n) \
  if constexpr (N == n) asm volatile("s_waitcnt vmcnt(" #n ") lgkmcnt(0)\n\ts_barrier" ::: "memory");
  SR_VMB_CASE(0) SR_VMB_CASE(1) SR_VMB_CASE(2) SR_VMB_CASE(3) SR_VMB_CASE(4) SR_VMB_CASE(5) SR_VMB_CASE(6)
  SR_VMB_CASE(7) SR_VMB_CASE(8) SR_VMB_CASE(9) SR_VMB_CASE(10) SR_VMB_CASE(11) SR_VMB_CASE(12)
  SR_VMB_CASE(13) SR_VMB_CASE(14) SR_VMB_CASE(15) SR_VMB_CASE(16) SR_VMB_CASE(17) SR_VMB_CASE(18)
  SR_VMB_CASE(19) SR_VMB_CASE(20) SR_VMB_CASE(21) SR_VMB_CASE(22) SR_VMB_CASE(23) SR_VMB_CASE(24)
  SR_VMB_CASE(25) SR_VMB_CASE(26) SR_VMB_CASE(27) SR_VMB_CASE(28) SR_VMB_CASE(29) SR_VMB_CASE(30)
  SR_VMB_CASE(31) SR_VMB_CASE(32) SR_VMB_CASE(33) SR_VMB_CASE(34) SR_VMB_CASE(35) SR_VMB_CASE(36)
  SR_VMB_CASE(37) SR_VMB_CASE(38) SR_VMB_CASE(39) SR_VMB_CASE(40) SR_VMB_CASE(41) SR_VMB_CASE(42)
  SR_VMB_CASE(43) SR_VMB_CASE(44) SR_VMB_CASE(45) SR_VMB_CASE(46) SR_VMB_CASE(47) SR_VMB_CASE(48)
  SR_VMB_CASE(49) SR_VMB_CASE(50) SR_VMB_CASE(51) SR_VMB_CASE(52) SR_VMB_CASE(53) SR_VMB_CASE(54)
  SR_VMB_CASE(55) SR_VMB_CASE(56) SR_VMB_CASE(57) SR_VMB_CASE(58) SR_VMB_CASE(59) SR_VMB_CASE(60)
  SR_VMB_CASE(61) SR_VMB_CASE(62) SR_VMB_CASE(63)
#undef SR_VMB_CASE
}
template <int D, int A>
__device__ __forceinline__ void vm_barrier_ahead(int a) {
  if constexpr (A <= 0) {
    vm_barrier<0>();
  } else {
    if (a >= A) vm_barrier<A * D>();
    else vm_barrier_ahead<D, A - 1>(a);
  }
}

// ------------------------------------- bf16 MFMA GEMM, few rows (LDS DMA)
// For the decode projections (a few hundred rows at most) the weights are
// streamed once from HBM; what matters is keeping enough of them in flight
// and keeping the per-step overhead small.  Block tile BM x BN (PAIRED: BN
// gate rows then BN up rows, BN output columns), K step BK (64, 128 or
// 256), NST LDS stages filled by global_load_lds_dwordx4 up to NST - 1 steps
// ahead, one barrier per step.  LDS stage: the BM activation rows then the
// weight rows, 2 BK bytes each; 16-byte chunk c of row r sits in slot
// c ^ (r & 15) (BK 128, 256) or c ^ (r & 7) ^ ((r >> 3) & 1) (BK 64), so the
// fragment reads of 16 consecutive rows are free of bank conflicts.  With
// rot > 0 tile n visits its K steps from step (n rot) mod nk on, wrapping
// around (the same products, summed in that order).  4 waves in a WGM x WGN
// grid, each a (BM / WGM) x (BN / WGN) tile of v_mfma_f32_16x16x32_bf16
// accumulators; the fragment reads of the next 32-wide sub-step run under
// the MFMAs of the current one.

template <int BK>
__device__ __forceinline__ int stream_slot(int c, int r) {
  if constexpr (BK >= 128) return c ^ (r & 15);
  else return c ^ (r & 7) ^ ((r >> 3) & 1);
}

// Epilogue of the few-row kernels.  The weight fragment is the first MFMA
// operand, so the accumulators hold the transposed tile: lane l has row
// mrow + 16 i and the four consecutive columns ncol + 16 j .. + 3, stored as
// one 16-byte (fp32) or 8-byte (bf16) chunk where the row is aligned and the
// columns are inside the output.
template <int NB, int TI, int TJ, bool PAIRED>
__device__ __forceinline__ void stream_epilogue(const f32x4 (&acc)[NB][TI][TJ], int mrow, int ncol, int M, int N,
                                                int split, const EpiArgs& epi, float* __restrict__ partial) {
  const bool to_part = partial != nullptr;
  const bool resid = !PAIRED && !to_part && epi.mode == EPI_RESID;
  const bool bf = !to_part && !resid && epi.out_bf16;
  const int64_t ld = to_part ? (int64_t)NB * N : (int64_t)epi.ldo;
  const bool aligned = to_part ? (N % 4 == 0 && (reinterpret_cast<uintptr_t>(partial) & 15) == 0)
                               : (epi.ldo % 4 == 0 && (reinterpret_cast<uintptr_t>(epi.out) & 15) == 0);
  float* const fbase = to_part ? partial + (int64_t)split * M * ld : reinterpret_cast<float*>(epi.out);
  bf16_t* const bbase = reinterpret_cast<bf16_t*>(epi.out);
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int m = mrow + 16 * i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int n = ncol + 16 * j;
      if (n >= N) continue;
      const bool full = aligned && n + 3 < N;
      const int64_t off = (int64_t)m * ld + n;
      f32x4 v = acc[0][i][j];
      if (to_part) {
        if (full) {
          store4(fbase + off, v);
          if (PAIRED) store4(fbase + off + N, acc[NB - 1][i][j]);
        } else {
          for (int k = 0; k < 4 && n + k < N; ++k) {
            fbase[off + k] = v[k];
            if (PAIRED) fbase[off + N + k] = acc[NB - 1][i][j][k];
          }
        }
        continue;
      }
      if (PAIRED) {
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = silu(v[k]) * acc[NB - 1][i][j][k];
      }
      if (full) {
        if (resid) v += *reinterpret_cast<const f32x4*>(fbase + off);
        if (bf) store4(bbase + off, v);
        else store4(fbase + off, v);
      } else {
        for (int k = 0; k < 4 && n + k < N; ++k) {
          if (resid) fbase[off + k] += v[k];
          else if (bf) bbase[off + k] = f32_to_bf16(v[k]);
          else fbase[off + k] = v[k];
        }
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN, int NST, bool PAIRED, int BK>
__global__ void __launch_bounds__(256)
gemm_stream_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb,
                   int64_t pair_off, int M, int N, int K, int k_per_split, int rot, EpiArgs epi,
                   float* __restrict__ partial) {
  constexpr int NB = PAIRED ? 2 : 1;
  constexpr int BNL = NB * BN;                  // weight rows per tile
  constexpr int ROWS = BM + BNL;
  constexpr int STAGE = ROWS * BK;              // bf16 elements per stage
  constexpr int CH = BK / 8;                    // 16-byte chunks per row
  constexpr int RPI = 64 / CH;                  // rows per DMA instruction (1 KB)
  constexpr int D = ROWS / (4 * RPI);           // DMA instructions per wave per stage
  constexpr int NS = BK / 32;                   // MFMA sub-steps per stage
  constexpr int WM = BM / WGM, WN = BN / WGN, TI = WM / 16, TJ = WN / 16;
  static_assert((BK == 64 || BK == 128 || BK == 256) && ROWS % (4 * RPI) == 0 && WGM * WGN == 4 && TI >= 1 &&
                    TJ >= 1 && NS % 2 == 0,
                "tile shape");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NST * STAGE];

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN - 1) / BN, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int m0 = tile.m * BM, n0 = tile.n * BN;
  const int k_begin = tile.split * k_per_split;
  const int nk = k_per_split / BK;
  const int s0 = rot > 0 ? (int)(((int64_t)tile.n * rot) % nk) : 0;

  // DMA instruction j covers tile rows RPI j .. RPI j + RPI - 1 (activation
  // rows first); wave w issues j = w + 4 q.  Lane l writes slot l % CH of
  // row l / CH and fetches the chunk stored there; rows past M or N are
  // clamped (their results are never stored).
  uint32_t off[D];
#pragma unroll
  for (int q = 0; q < D; ++q) {
    const int r = RPI * (wave + 4 * q) + lane / CH;
    const int c = stream_slot<BK>(lane % CH, r);
    int64_t e;
    if (r < BM) {
      e = (int64_t)min(m0 + r, M - 1) * lda;
    } else {
      const int rb = r - BM, blk = rb / BN;
      e = blk * pair_off + (int64_t)min(n0 + rb - blk * BN, N - 1) * ldb;
    }
    off[q] = (uint32_t)((e + c * 8) * 2);
  }
  const char* Ab = reinterpret_cast<const char*>(A + k_begin);
  const char* Bb = reinterpret_cast<const char*>(B + k_begin);
  auto issue = [&](int st, int buf) {
    bf16_t* dst = lds + buf * STAGE;
    const int k = st + s0;
    const int kb = (k >= nk ? k - nk : k) * BK * 2;
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const bool is_a = RPI * (wave + 4 * q) < BM;  // wave-uniform
      dma16((is_a ? Ab : Bb) + kb + off[q], dst + (wave + 4 * q) * 512);
    }
  };

  // 16x16x32 fragments: lane l holds row l % 16 of a 16-row block, K chunk
  // 4 s + l / 16 of sub-step s.
  const int fr = lane & 15, fg = lane >> 4;
  int foff[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) foff[s] = fr * BK + 8 * stream_slot<BK>(4 * s + fg, fr);

  f32x4 acc[NB][TI][TJ];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[b][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto read_frags = [&](const bf16_t* base, int s, bf16x8(&af)[TI], bf16x8(&bfr)[NB][TJ]) {
#pragma unroll
    for (int i = 0; i < TI; ++i) af[i] = *reinterpret_cast<const bf16x8*>(base + foff[s] + (wm0 + 16 * i) * BK);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        bfr[b][j] = *reinterpret_cast<const bf16x8*>(base + foff[s] + (BM + b * BN + wn0 + 16 * j) * BK);
  };
  auto mfma = [&](const bf16x8(&af)[TI], const bf16x8(&bfr)[NB][TJ]) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[b][j], af[i], acc[b][i][j], 0, 0, 0);
  };
  // one MFMA, then one fragment read of the next sub-step, alternating;
  // then the remaining MFMAs
  constexpr int NMF = NB * TI * TJ, NRD = TI + NB * TJ;
  auto interleave = [] {
#pragma unroll
    for (int k = 0; k < (NRD < NMF ? NRD : NMF); ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (NRD > NMF) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NMF, 0);
    if constexpr (NMF > NRD) __builtin_amdgcn_sched_group_barrier(0x008, NMF - NRD, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // Only steps that exist are fetched (a copy past the end would be waited
  // for before the work-group may end, a DMA round trip on every launch).
  for (int st = 0; st < NST - 1 && st < nk; ++st) issue(st, st);
  for (int t = 0; t < nk; ++t) {
    // step t landed; every wave is done with step t - 1's buffer: all but
    // the copies of the steps issued after t (NST - 2 of them, fewer at the
    // end).
    vm_barrier_ahead<D, NST - 2>(min(NST - 2, nk - 1 - t));
    if (t + NST - 1 < nk) issue(t + NST - 1, (t + NST - 1) % NST);
    const bf16_t* base = lds + (t % NST) * STAGE;
    bf16x8 a0[TI], b0[NB][TJ], a1[TI], b1[NB][TJ];
    read_frags(base, 0, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < NS; s += 2) {
      read_frags(base, s + 1, a1, b1);
      mfma(a0, b0);
      interleave();
      if (s + 2 < NS) {
        read_frags(base, s + 2, a0, b0);
        mfma(a1, b1);
        interleave();
      }
    }
    mfma(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
  }
  // no DMA may still be writing LDS when the work-group ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  stream_epilogue<NB, TI, TJ, PAIRED>(acc, m0 + wm0 + fr, n0 + wn0 + 4 * fg, M, N, tile.split, epi, partial);
}

// ------------------- bf16 MFMA GEMM, few rows, separate activation and weight rings
// The few-row kernel above with one LDS ring for the activation rows (read
// by every tile, resident in L2) and another for the weight rows (streamed
// once from HBM): NA activation stages filled one step ahead and NW weight
// stages filled NW - 1 steps ahead, so with 112 activation rows two weight
// stages are in flight where a shared ring of the same size holds one.  The
// copies of a step go out activation rows first, then weight rows; at step
// t the wait leaves in flight only the weight copies issued after the
// activation rows of step t (those of step t + NW - 2).  `rot` > 0 starts
// tile n at K step (n rot) mod nk and wraps, so the tiles stream their rows
// at staggered K offsets instead of in lockstep.  Fragment reads and the MFMA
// tiling are those of gemm_stream_kernel; BK 128 or 256 (a copy instruction
// then moves 4 rows of 256 bytes or 2 rows of 512 bytes).
template <int BM, int BN, int WGM, int WGN, int NA, int NW, bool PAIRED, int BK>
__global__ void __launch_bounds__(256)
gemm_ring_kernel(const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ B, int ldb, int64_t pair_off,
                 int M, int N, int K, int k_per_split, int rot, EpiArgs epi, float* __restrict__ partial) {
  constexpr int NB = PAIRED ? 2 : 1;
  constexpr int BNL = NB * BN;                  // weight rows per tile
  constexpr int CH = BK / 8;                    // 16-byte chunks per row
  constexpr int RPI = 64 / CH;                  // rows per copy instruction (1 KB)
  constexpr int DA = BM / (4 * RPI), DW = BNL / (4 * RPI);  // copies per wave per step
  constexpr int NS = BK / 32;                   // MFMA sub-steps per step
  constexpr int WM = BM / WGM, WN = BN / WGN, TI = WM / 16, TJ = WN / 16;
  constexpr int ASZ = BM * BK, WSZ = BNL * BK;  // bf16 elements per stage
  static_assert((BK == 128 || BK == 256) && BM % (4 * RPI) == 0 && BNL % (4 * RPI) == 0 && WGM * WGN == 4 &&
                    TI >= 1 && TJ >= 1 && NA >= 2 && NW >= 3 && NS % 2 == 0,
                "tile shape");
  static_assert((NA * ASZ + NW * WSZ) * 2 <= 160 * 1024, "LDS");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NA * ASZ + NW * WSZ];

  const TileIdx tile = tile_of((M + BM - 1) / BM, (N + BN - 1) / BN, K / k_per_split);
  if (!tile.valid) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int m0 = tile.m * BM, n0 = tile.n * BN;
  const int k_begin = tile.split * k_per_split;
  const int nk = k_per_split / BK;
  const int s0 = rot > 0 ? (int)(((int64_t)tile.n * rot) % nk) : 0;

  // Copy q of a wave moves rows RPI (wave + 4 q) .. + RPI - 1 of its ring
  // stage; lane l writes slot l % CH of row l / CH and fetches the chunk
  // stored there.  Rows past M or N are clamped (never stored).
  uint32_t aoff[DA], woff[DW];
#pragma unroll
  for (int q = 0; q < DA; ++q) {
    const int r = RPI * (wave + 4 * q) + lane / CH;
    const int c = stream_slot<BK>(lane % CH, r);
    aoff[q] = (uint32_t)(((int64_t)min(m0 + r, M - 1) * lda + c * 8) * 2);
  }
#pragma unroll
  for (int q = 0; q < DW; ++q) {
    const int rb = RPI * (wave + 4 * q) + lane / CH;
    const int c = stream_slot<BK>(lane % CH, rb);
    const int blk = rb / BN;
    woff[q] = (uint32_t)((blk * pair_off + (int64_t)min(n0 + rb - blk * BN, N - 1) * ldb + c * 8) * 2);
  }
  const char* Ab = reinterpret_cast<const char*>(A + k_begin);
  const char* Bb = reinterpret_cast<const char*>(B + k_begin);
  bf16_t* const wring = lds + NA * ASZ;
  // byte offset of step st's K columns
  auto kbyte = [&](int st) {
    const int k = st + s0;
    return (k >= nk ? k - nk : k) * BK * 2;
  };
  auto issue_a = [&](int st, int buf) {
    bf16_t* dst = lds + buf * ASZ;
    const int kb = kbyte(st);
#pragma unroll
    for (int q = 0; q < DA; ++q) dma16(Ab + kb + aoff[q], dst + (wave + 4 * q) * 512);
  };
  auto issue_w = [&](int st, int buf) {
    bf16_t* dst = wring + buf * WSZ;
    const int kb = kbyte(st);
#pragma unroll
    for (int q = 0; q < DW; ++q) dma16(Bb + kb + woff[q], dst + (wave + 4 * q) * 512);
  };

  const int fr = lane & 15, fg = lane >> 4;
  int foff[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) foff[s] = fr * BK + 8 * stream_slot<BK>(4 * s + fg, fr);

  f32x4 acc[NB][TI][TJ];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[b][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto read_frags = [&](const bf16_t* ab, const bf16_t* wb, int s, bf16x8(&af)[TI], bf16x8(&bfr)[NB][TJ]) {
#pragma unroll
    for (int i = 0; i < TI; ++i) af[i] = *reinterpret_cast<const bf16x8*>(ab + foff[s] + (wm0 + 16 * i) * BK);
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        bfr[b][j] = *reinterpret_cast<const bf16x8*>(wb + foff[s] + (b * BN + wn0 + 16 * j) * BK);
  };
  auto mfma = [&](const bf16x8(&af)[TI], const bf16x8(&bfr)[NB][TJ]) {
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[b][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[b][j], af[i], acc[b][i][j], 0, 0, 0);
  };
  constexpr int NMF = NB * TI * TJ, NRD = TI + NB * TJ;
  auto interleave = [] {
#pragma unroll
    for (int k = 0; k < (NRD < NMF ? NRD : NMF); ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if constexpr (NRD > NMF) __builtin_amdgcn_sched_group_barrier(0x100, NRD - NMF, 0);
    if constexpr (NMF > NRD) __builtin_amdgcn_sched_group_barrier(0x008, NMF - NRD, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // Prologue: activation rows of step 0, weight rows of steps 0 .. NW - 2
  // (only steps that exist: a copy past the end would be waited for before
  // the work-group may end).
  issue_a(0, 0);
  for (int st = 0; st < NW - 1 && st < nk; ++st) issue_w(st, st);
  for (int t = 0; t < nk; ++t) {
    // Steps t of both rings landed, and every wave is done with the buffers
    // of step t - 1 (refilled below).  Issued after the activation rows of
    // step t: at t = 0 the weight rows of steps 1 .. NW - 2; later those of
    // step t + NW - 2 (issued with them at step t - 1), when it exists.
    if (t == 0) vm_barrier_ahead<DW, NW - 2>(min(NW - 2, nk - 1));
    else vm_barrier_ahead<DW, 1>(t + NW - 2 < nk ? 1 : 0);
    if (t + 1 < nk) issue_a(t + 1, (t + 1) % NA);
    if (t + NW - 1 < nk) issue_w(t + NW - 1, (t + NW - 1) % NW);
    const bf16_t* ab = lds + (t % NA) * ASZ;
    const bf16_t* wb = wring + (t % NW) * WSZ;
    bf16x8 a0[TI], b0[NB][TJ], a1[TI], b1[NB][TJ];
    read_frags(ab, wb, 0, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < NS; s += 2) {
      read_frags(ab, wb, s + 1, a1, b1);
      mfma(a0, b0);
      interleave();
      if (s + 2 < NS) {
        read_frags(ab, wb, s + 2, a0, b0);
        mfma(a1, b1);
        interleave();
      }
    }
    mfma(a1, b1);
    __builtin_amdgcn_sched_barrier(0);
  }
  // no DMA may still be writing LDS when the work-group ends
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  stream_epilogue<NB, TI, TJ, PAIRED>(acc, m0 + wm0 + fr, n0 + wn0 + 4 * fg, M, N, tile.split, epi, partial);
}

// ------------------------------------------------------------ fp32 GEMM
// 64 x 64 block tile, 256 threads, 4 x 4 outputs per thread, K step 16.
// Always writes to `partial` ([1][M][NB*N]); the reduce kernel applies the
// epilogue.
__global__ void __launch_bounds__(256)
gemm_f32_kernel(const float* __restrict__ A, int lda, const float* __restrict__ B, int ldb,
                int64_t pair_off, int paired, int M, int N, int K, float* __restrict__ partial) {
  __shared__ float As[16][64 + 1];
  __shared__ float Bs[16][64 + 1];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int m0 = blockIdx.y * 64;
  const int nb = paired ? 2 : 1;
  const int ncols = nb * N;
  const int n0 = blockIdx.x * 64;  // over the concatenated [gate | up] columns
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int c = tid; c < 64 * 16; c += 256) {
      int r = c / 16, kk = c % 16;
      int m = m0 + r, n = n0 + r;
      As[kk][r] = (m < M) ? A[(int64_t)m * lda + k0 + kk] : 0.f;
      float bv = 0.f;
      if (n < ncols) {
        int blk = n / N, nn = n % N;
        bv = B[blk * pair_off + (int64_t)nn * ldb + k0 + kk];
      }
      Bs[kk][r] = bv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      if (m < M && n < ncols) partial[(int64_t)m * ncols + n] = acc[i][j];
    }
}

// Sum split-K partials in split order, then apply the epilogue.
__global__ void gemm_reduce_kernel(const float* __restrict__ partial, int splits, int M, int N,
                                   int paired, EpiArgs epi) {
  const int nout = paired ? 2 * N : N;
  const int64_t total = (int64_t)M * N;
  for (int64_t idx = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int m = (int)(idx / N), n = (int)(idx % N);
    float g = 0.f, u = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float* p = partial + ((int64_t)s * M + m) * nout;
      g += p[n];
      if (paired) u += p[N + n];
    }
    if (paired)
      store_out(epi, m, n, silu(g) * u);
    else
      epi_one(epi, m, n, g);
  }
}

// ------------------------------------------------------------ dispatch
template <int BM, int BN, int BK, int WM, int WN, bool PAIRED>
static void launch_bf16(const GemmArgs& g, int splits, int kps, const EpiArgs& e, float* part,
                        hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  dim3 grid = tile_grid((g.M + BM - 1) / BM, (g.N + BN - 1) / BN, splits);
  SR_LAUNCH((gemm_bf16_kernel<BM, BN, BK, WM, WN, PAIRED>), grid, dim3(NT), 0, s,
                     (const bf16_t*)g.A, g.lda, (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N,
                     g.K, kps, e, part);
  SR_CHECK_LAUNCH();
}

size_t gemm_partial_elems(int dtype, int M, int N, int K, bool paired) {
  GemmPlan p = gemm_plan(dtype, M, N, K, paired);
  if (p.splits <= 1 && dtype == SR_BF16) return 0;
  return (size_t)p.splits * M * (paired ? 2 * (size_t)N : (size_t)N);
}

// Partials needed by an EPI_PARTIAL call (written even without a K split).
size_t gemm_partial_elems_always(int dtype, int M, int N, int K) {
  GemmPlan p = gemm_plan(dtype, M, N, K, false);
  return (size_t)p.splits * M * (size_t)N;
}

// Dispatch thresholds (rows M of the projection), measured on MI355X:
//  - up to kStreamMaxRows rows the LDS-DMA streaming kernel (weights read
//    once, one work-group per CU);
//  - up to kDma3MaxRows rows the 256 x 256 tile with the three-deep weight
//    ring when its grid holds at least kDmaWideMinTiles tiles, else the
//    three-stage 256 x 128 tile;
//  - from kDmaMinRows rows (or 256 rows with kDmaWideMinTiles tiles) the
//    LDS-DMA 256 x 256 tile, and the register-staged 256 x 256 tile when
//    an operand is too large for 32-bit buffer offsets.
constexpr int kStreamMaxRows = 128;
constexpr int kDma3MaxRows = 512;
constexpr int kDmaWideMinTiles = 192;
constexpr int kDmaMinRows = 1024;
constexpr int kBigTileMinRows = 1024;
constexpr int kTileRot = 7;

static int stream_tile_rows(int M) { return M <= 32 ? 32 : (M <= 64 ? 64 : (M <= 112 ? 112 : 128)); }

GemmPlan gemm_plan(int dtype, int M, int N, int K, bool paired) {
  GemmPlan p;
  p.splits = 1;
  p.big = false;
  p.dma = false;
  p.dma3 = false;
  p.dma_bring = 2;
  p.stream = 0;
  p.stream_bn = 0;
  if (dtype != SR_BF16) return p;
  if (M > 64 && M <= 112 && !paired && N > 65536 && K % 128 == 0) {
    // The LM head at 65-112 rows: 112 x 128 tiles, one per work-group, with
    // the separate activation and weight rings (enough tiles without split).
    p.stream = 112;
    p.stream_bn = 128;
    return p;
  }
  if (M <= kStreamMaxRows && K % 128 == 0 && (M <= 64 || N <= 65536)) {
    // One round of work-groups (one per CU): split K by the largest power of
    // two that keeps the grid within 256 and each split a multiple of 128.
    p.stream = stream_tile_rows(M);
    p.stream_bn = 64;
    const int64_t tiles = (int64_t)((M + p.stream - 1) / p.stream) * ((N + p.stream_bn - 1) / p.stream_bn);
    int splits = 1;
    while (tiles * splits * 2 <= 256 && K % (splits * 2 * 128) == 0) splits *= 2;
    p.splits = splits;
    return p;
  }
  if (M > kStreamMaxRows && M <= kDma3MaxRows && K % 64 == 0) {
    // A few hundred rows, a grid of 256 x 256 tiles that alone fills most of
    // the CUs: that tile with the three-deep weight ring, unsplit.
    const int64_t wide = (int64_t)((M + 255) / 256) * ((N + (paired ? 127 : 255)) / (paired ? 128 : 256));
    if (wide >= kDmaWideMinTiles) {
      p.dma = true;
      p.dma_bring = 3;
      return p;
    }
    // Otherwise (the first decode round) 256 x 128 tiles with three stages;
    // split K (each split a multiple of 64 and at least 512 long) by powers
    // of two while the grid stays within 256.
    p.dma3 = true;
    const int64_t tiles = (int64_t)((M + 255) / 256) * ((N + (paired ? 63 : 127)) / (paired ? 64 : 128));
    int splits = 1;
    while (tiles * splits * 2 <= 256 && K % (splits * 2 * 64) == 0 && K / (splits * 2) >= 512) splits *= 2;
    p.splits = splits;
    return p;
  }
  const int64_t dma_tiles = (int64_t)((M + 255) / 256) * ((N + (paired ? 127 : 255)) / (paired ? 128 : 256));
  if (K % 64 == 0 && (M >= kDmaMinRows || (M >= 256 && dma_tiles >= kDmaWideMinTiles))) {
    // One work-group per CU at least: split K (each split a multiple of 64
    // and at least 512 long) while the tile grid is smaller than 256.
    p.dma = true;
    const int64_t tiles = dma_tiles;
    int splits = 1;
    while (tiles * splits < 256 && K % (splits * 2 * 64) == 0 && K / (splits * 2) >= 512 && splits < 8)
      splits *= 2;
    p.splits = splits;
    return p;
  }
  if (M >= kBigTileMinRows) {
    p.big = true;
    return p;
  }
  int bm = M <= 32 ? 32 : (M <= 64 ? 64 : 128);
  int bn = paired ? 64 : 128;
  int64_t tiles = (int64_t)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  // Split K when the tile grid alone cannot fill 256 CUs twice over; each
  // split keeps at least 512 of K and a multiple of 64.
  int splits = 1;
  while (tiles * splits < 512 && K % (splits * 2 * 64) == 0 && K / (splits * 2) >= 512 && splits < 8)
    splits *= 2;
  p.splits = splits;
  return p;
}

// The LDS-DMA kernels address their operands with 32-bit byte offsets from
// the K base of the split; the tiled ones pass them to buffer loads as signed
// 32-bit vector offsets, so there they stay below 2 GiB (larger operands take
// the register-staged kernels).
static bool dma_offsets_fit(const GemmArgs& g, int bits = 32) {
  const int64_t a = ((int64_t)(g.M - 1) * g.lda + g.K) * 2;
  const int64_t b = ((g.paired ? g.pair_off : 0) + (int64_t)(g.N - 1) * g.ldb + g.K) * 2;
  return a < (1LL << bits) && b < (1LL << bits) && g.pair_off >= 0;
}

int gemm(const GemmArgs& g, float* partial, size_t partial_cap, hipStream_t s) {
  SR_REQUIRE(g.K % 64 == 0, 3, "GEMM K must be a multiple of 64");
  SR_REQUIRE(!(g.epi == EPI_PARTIAL && g.paired), 5, "partial epilogue is for unpaired projections");
  EpiArgs e{g.epi, g.out, g.ldo, g.out_bf16};
  if (g.M == 0 || g.N == 0) return 1;
  if (g.dtype == SR_F32) {
    const int ncols = (g.paired ? 2 : 1) * g.N;
    SR_REQUIRE((size_t)g.M * ncols <= partial_cap, 5, "GEMM partial buffer too small");
    dim3 grid((ncols + 63) / 64, (g.M + 63) / 64);
    SR_LAUNCH(gemm_f32_kernel, grid, dim3(256), 0, s, (const float*)g.A, g.lda,
                       (const float*)g.B, g.ldb, g.pair_off, (int)g.paired, g.M, g.N, g.K, partial);
    SR_CHECK_LAUNCH();
    if (g.epi == EPI_PARTIAL) return 1;
    int64_t total = (int64_t)g.M * g.N;
    int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
    SR_LAUNCH(gemm_reduce_kernel, dim3(blocks), dim3(256), 0, s, partial, 1, g.M, g.N,
                       (int)g.paired, e);
    SR_CHECK_LAUNCH();
    return 1;
  }
  GemmPlan plan = gemm_plan(g.dtype, g.M, g.N, g.K, g.paired);
  const int splits = plan.splits;
  const int kps = g.K / splits;
  SR_REQUIRE(kps * splits == g.K && kps % 64 == 0, 5, "split-K must divide K into multiples of 64");
  float* part = nullptr;
  if (splits > 1 || g.epi == EPI_PARTIAL) {
    SR_REQUIRE((size_t)splits * g.M * (g.paired ? 2 : 1) * (size_t)g.N <= partial_cap, 5,
               "GEMM partial buffer too small");
    part = partial;
  }
  if (plan.stream && dma_offsets_fit(g)) {
    dim3 grid = tile_grid((g.M + plan.stream - 1) / plan.stream, (g.N + plan.stream_bn - 1) / plan.stream_bn, splits);
#define SR_STREAM(BM, BN, WGM, WGN, NST, P, BK, ROT)                                                    \
  SR_LAUNCH((gemm_stream_kernel<BM, BN, WGM, WGN, NST, P, BK>), grid, dim3(256), 0, s,           \
                     (const bf16_t*)g.A, g.lda, (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, ROT, e, \
                     part)
#define SR_RING(BM, BN, WGM, WGN, NA, NW, P, BK, ROT)                                                    \
  SR_LAUNCH((gemm_ring_kernel<BM, BN, WGM, WGN, NA, NW, P, BK>), grid, dim3(256), 0, s,          \
                     (const bf16_t*)g.A, g.lda, (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, ROT, e, \
                     part)
    // The paired (gate and up) projections start each tile at its own K
    // step (rotation kTileRot); without it their tiles stream both weight
    // blocks in lockstep and reach 4.0-4.4 TB/s, with it 5.0-5.7 (measured
    // on the 8B shapes at 21-128 rows).
    if (plan.stream == 32) {
      if (g.paired) {
        // 2 rows of 512 bytes per copy instruction
        if (kps % 256 == 0) SR_STREAM(32, 64, 1, 4, 2, true, 256, kTileRot);
        else SR_STREAM(32, 64, 1, 4, 3, true, 128, kTileRot);
      } else {
        SR_STREAM(32, 64, 1, 4, 5, false, 128, 0);
      }
    } else if (plan.stream == 64) {
      if (g.paired) SR_STREAM(64, 64, 2, 2, 3, true, 128, kTileRot);
      else SR_STREAM(64, 64, 2, 2, 4, false, 128, 0);
    } else if (plan.stream == 112) {
      // 65-112 rows: seven 16-row blocks per wave, the four waves side by
      // side over the columns (less padding than 128 rows); paired: two
      // weight stages in flight beside the activation ring
      if (g.paired) SR_RING(112, 64, 1, 4, 2, 3, true, 128, kTileRot);
      else if (plan.stream_bn == 128) SR_RING(112, 128, 1, 4, 2, 3, false, 128, 0);
      else SR_STREAM(112, 64, 1, 4, 3, false, 128, 0);
    } else {
      if (g.paired) SR_RING(128, 64, 2, 2, 2, 3, true, 128, kTileRot);
      else SR_STREAM(128, 64, 2, 2, 3, false, 128, 0);
    }
#undef SR_RING
#undef SR_STREAM
    SR_CHECK_LAUNCH();
  } else if (plan.dma3 && dma_offsets_fit(g, 31)) {
    const int bn_out = g.paired ? 64 : 128;
    dim3 grid = tile_grid((g.M + 255) / 256, (g.N + bn_out - 1) / bn_out, splits);
    if (g.paired)
      SR_LAUNCH(gemm_dma3_kernel<true>, grid, dim3(256), 0, s, (const bf16_t*)g.A, g.lda,
                         (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, e, part);
    else
      SR_LAUNCH(gemm_dma3_kernel<false>, grid, dim3(256), 0, s, (const bf16_t*)g.A, g.lda,
                         (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, e, part);
    SR_CHECK_LAUNCH();
  } else if (plan.dma && dma_offsets_fit(g, 31)) {
    const int bn_out = g.paired ? 128 : 256;
    dim3 grid = tile_grid((g.M + 255) / 256, (g.N + bn_out - 1) / bn_out, splits);
#define SR_DMA(P, R)                                                                                   \
  SR_LAUNCH((gemm_dma_kernel<P, R>), grid, dim3(256), 0, s, (const bf16_t*)g.A, g.lda,        \
                     (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, e, part)
    if (plan.dma_bring == 3) {
      if (g.paired) SR_DMA(true, 3);
      else SR_DMA(false, 3);
    } else {
      if (g.paired) SR_DMA(true, 2);
      else SR_DMA(false, 2);
    }
#undef SR_DMA
    SR_CHECK_LAUNCH();
  } else if (plan.big || plan.dma) {
    const int bn_out = g.paired ? 128 : 256;
    dim3 grid = tile_grid((g.M + 255) / 256, (g.N + bn_out - 1) / bn_out, splits);
    if (g.paired)
      SR_LAUNCH(gemm_big_kernel<true>, grid, dim3(256), 0, s, (const bf16_t*)g.A, g.lda,
                         (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, e, part);
    else
      SR_LAUNCH(gemm_big_kernel<false>, grid, dim3(256), 0, s, (const bf16_t*)g.A, g.lda,
                         (const bf16_t*)g.B, g.ldb, g.pair_off, g.M, g.N, g.K, kps, e, part);
    SR_CHECK_LAUNCH();
  } else if (g.paired) {
    if (g.M <= 32) launch_bf16<32, 64, 64, 32, 16, true>(g, splits, kps, e, part, s);
    else if (g.M <= 64) launch_bf16<64, 64, 64, 32, 32, true>(g, splits, kps, e, part, s);
    else launch_bf16<128, 64, 64, 64, 32, true>(g, splits, kps, e, part, s);
  } else {
    if (g.M <= 32) launch_bf16<32, 128, 64, 32, 32, false>(g, splits, kps, e, part, s);
    else if (g.M <= 64) launch_bf16<64, 128, 64, 32, 64, false>(g, splits, kps, e, part, s);
    else launch_bf16<128, 128, 64, 64, 64, false>(g, splits, kps, e, part, s);
  }
  if (splits > 1 && g.epi != EPI_PARTIAL) {
    int64_t total = (int64_t)g.M * g.N;
    int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    SR_LAUNCH(gemm_reduce_kernel, dim3(blocks), dim3(256), 0, s, part, splits, g.M, g.N,
                       (int)g.paired, e);
    SR_CHECK_LAUNCH();
  }
  return splits;
}

}  // namespace sr
