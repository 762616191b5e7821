// Launchers of the device kernels (all asynchronous on the given stream).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/specrej.h"

namespace sr {

// ---- GEMM -------------------------------------------------------------------
enum GemmEpi { EPI_STORE = 0, EPI_RESID = 1, EPI_PARTIAL = 2 };

struct GemmArgs {
  int dtype;             // SR_F32 / SR_BF16: element type of A and B
  const void* A;         // [M][lda] activations
  int lda;
  const void* B;         // [N][ldb] weights (second block at B + pair_off when paired)
  int ldb;
  int64_t pair_off;      // elements between the gate and up blocks (paired only)
  bool paired;           // out = silu(A B_gate^T) * (A B_up^T)
  int M, N, K;
  int epi;               // EPI_STORE (out = C), EPI_RESID (fp32 out += C) or EPI_PARTIAL
                         // (fp32 split partials [splits][M][N] left in `partial` for a
                         // fused consumer; gemm() returns the split count); paired: store
  void* out;
  int ldo;
  int out_bf16;          // EPI_STORE / paired: 1 = bf16 out, 0 = fp32 out
};
struct GemmPlan {
  int splits;
  bool big;     // 256 x 256 tile kernel
  bool dma;     // 256 x 256 tile fed by LDS DMA
  int dma_bring;  // its weight ring depth: 2 (shared with the activations) or 3
  bool dma3;    // 256 x 128 tile, three LDS-DMA stages (a few hundred rows)
  int stream;     // > 0: LDS-DMA streaming kernel for few rows, tile height
  int stream_bn;  // its tile width (output columns)
};
GemmPlan gemm_plan(int dtype, int M, int N, int K, bool paired);
size_t gemm_partial_elems(int dtype, int M, int N, int K, bool paired);
int gemm(const GemmArgs& g, float* partial, size_t partial_cap, hipStream_t s);
size_t gemm_partial_elems_always(int dtype, int M, int N, int K);

// ---- elementwise / small ------------------------------------------------------
// h[r][:] = float(E[tok[r]][:]), r < rows.
void embed(int dtype, const void* E, int d, const int32_t* tok, int rows, float* h, hipStream_t s);
// out[r][:] = x[r][:] / sqrt(mean(x^2) + eps) * g, out in the model dtype.
void rmsnorm(int dtype, const float* x, int ldx, const void* g, int d, float eps, int rows, void* out,
             int ldo, hipStream_t s);
// tab[p][i] = (cos, sin)(p * theta^(-2i/hd)), p < npos, evaluated in double.
void rope_table(float2* tab, int npos, int hd, double theta, hipStream_t s);
// RoPE + scatter of a QKV projection for `rows` rows of `lr` tokens each:
// token (r, t) at position pos0 + t; q -> qout[(r*lr+t)][hq][hd] (fp32);
// k, v -> kdst/vdst[r][hkv][cap][hd] at token t0 + t (model dtype).
void rope_scatter(int dtype, const float* qkv, int rows, int lr, int hq, int hkv, int hd,
                  const float2* tab, int pos0, float* qout, void* kdst, void* vdst, int cap,
                  int t0, hipStream_t s);
// score[r] = w . RMSNorm(h[r*lr + len[r]-1-t0]) * g  (fused reward head;
// h holds response positions t0..t0+lr-1 of each row, t0 < len[r] <= t0+lr).
void score_head(int dtype, const float* h, int d, int lr, int t0, const int32_t* len, int rows,
                const void* g, const void* w, float eps, float* score, hipStream_t s);
// tokens[r][t] = t0+t < len[r] ? store[cand[r]][t0+t] : 0 for t < lr (store row stride ld).
void gather_tokens(const int32_t* store, int ld, const int32_t* cand, const int32_t* len, int rows,
                   int t0, int lr, int32_t* tokens, hipStream_t s);
void philox_fill(uint64_t seed, const uint32_t* ctr, int n, uint32_t* out, hipStream_t s);
// h[r] = E[tok[r]] (fp32); xn[r] = RMSNorm(h[r]) * g (model dtype).
void embed_norm(int dtype, const void* E, int d, const int32_t* tok, int rows, const void* g, float eps,
                float* h, void* xn, hipStream_t s);
// h[r] += sum_s part[s][r]; xn[r] = RMSNorm(h[r]) * g (model dtype); d columns.
void add_norm(int dtype, const float* part, int splits, int rows, int d, float* h, const void* g, float eps,
              void* xn, hipStream_t s);
// qkv[r] = sum_s part[s][r] (rows of (hq + 2 hkv) hd); RoPE at position pos
// on q and k; q -> qout[r][hq][hd] (fp32); k, v -> kdst/vdst[r][hkv][cap][hd]
// at token t0.
void qkv_finalize(int dtype, const float* part, int splits, int rows, int hq, int hkv, int hd,
                  const float2* tab, int pos, float* qout, void* kdst, void* vdst, int cap, int t0,
                  hipStream_t s);

// ---- attention ----------------------------------------------------------------
// Decode: one query per row at the newest position.  Keys: the shared prefix
// kpre/vpre [hkv][P][hd] then the row's tail ktail/vtail [row][hkv][cap][hd]
// of length lt.  q fp32 [rows][hq][hd]; out [rows][hq*hd] (model dtype).
struct DecodeAttnArgs {
  int dtype, hd, hq, hkv, rows;
  const float* q;
  const void *kpre, *vpre;
  int P;
  const void *ktail, *vtail;
  int cap, lt;
  void* out;
  float* part;       // split partials [rows][hq][splits][hd + 2]
  size_t part_cap;   // floats
  // Fused QKV finalize (decode_attn_fuses_qkv): instead of q, the QKV
  // projection's split partials qpart [qsplits][rows][qkv_dim] are summed
  // here; q and k heads are rotated with rope[hd / 2] (the table row of the
  // new position); the new K/V row is written to ktail/vtail at index lt - 1
  // before it is attended, and the rotated fp32 q to qout (for the prefix
  // pass) when qout is set.
  const float* qpart = nullptr;
  int qsplits = 0, qkv_dim = 0;
  const float2* rope = nullptr;
  float* qout = nullptr;
};
int decode_attn_splits(int rows, int hkv, int keys);
bool decode_attn_fuses_qkv(const DecodeAttnArgs& a);
void decode_attn(const DecodeAttnArgs& a, hipStream_t s);
// Partial floats decode_attn writes for these arguments (0 when it needs none).
size_t decode_attn_part_floats(const DecodeAttnArgs& a);
// The file-scope scratch array of the no-allocation decode attention: its
// size in floats, and its address on the current device (looked up once per
// device).
constexpr size_t kStaticScratchFloats = (size_t)8 << 20;  // 32 MiB
constexpr int kMaxDevices = 64;
float* static_scratch_of_current_device();

// Prefill: rows of lr new tokens that follow t0 tokens already cached for
// their row; new token (r, t) sits at response position t0 + t and attends
// the shared prefix kpre/vpre [hkv][P][hd] and its row's own keys
// 0..t0 + t in kown/vown [r][hkv][cap][hd] (cap >= t0 + lr).
// q fp32 [rows*lr][hq][hd]; out [rows*lr][hq*hd].
struct PrefillAttnArgs {
  int dtype, hd, hq, hkv, rows, lr;
  const float* q;
  const void *kpre, *vpre;
  int P;
  const void *kown, *vown;
  int cap = 0, t0 = 0;
  void* out;
};
void prefill_attn(const PrefillAttnArgs& a, hipStream_t s);

// ---- sampling and state ------------------------------------------------------
// For each row r with done[r] == 0: draw a token from logits row
// (broadcast ? 0 : r) keyed by (seed, cand[r], step); write it to
// store[cand[r]][step] and next_tok[r]; set done[r] if it equals eos_id;
// len[r] = step + 1.  done/len/store may be null (kernel-level entry).
struct SampleArgs {
  const float* logits;
  int64_t row_stride;    // 0 = every row reads row 0
  int rows, vocab;
  const int32_t* cand;
  int step;
  float temperature;
  uint64_t seed;
  int32_t* next_tok;
  int32_t* done;
  int32_t* len;
  int32_t* store;
  int store_ld;
  int eos_id;
};
void sample(const SampleArgs& a, hipStream_t s);

// Probability-as-reward (section 5.3): for every row sampled at `step`
// (len[r] == step + 1), lp_sum[cand[r]] += ln softmax(logits row)[tok[r]]
// at temperature 1 (fixed-order fp32 reductions).
void logprob_accumulate(const float* logits, int64_t row_stride, int rows, int vocab, const int32_t* cand,
                        const int32_t* tok, const int32_t* len, int step, float* lp_sum, hipStream_t s);
// score[r] = lp_sum[cand[r]] / len[r] (0 for an empty response).
void logprob_scores(const float* lp_sum, const int32_t* cand, const int32_t* len, int rows, float* score,
                    hipStream_t s);

// ---- the cut ------------------------------------------------------------------
// accept[i] = rank of (score[i] desc, cand[i] asc, NaN lowest) < keep.
void select_topk(const float* score, const int32_t* cand, int b, int keep, int32_t* accept,
                 hipStream_t s);
// Full cut for the generation loop (single work-group, b <= 4096):
// ranks, accept flags, completed rows appended to I, and the packed state of
// the kept unfinished rows: src_row[j], cand_out/len_out/tok_out[j], count.
struct CutArgs {
  const float* score;
  const int32_t *cand, *len, *done, *next_tok;
  int b, keep;
  int32_t* accept;                    // [b]
  int32_t *i_cand, *i_len, *i_count;  // set I (append)
  float* i_score;
  int32_t *src_row, *cand_out, *len_out, *tok_out, *count;
};
void cut(const CutArgs& a, hipStream_t s);
// Packs kept rows (keep_flag != 0, or the first *count entries of src_row
// when keep_flag is null) of a KV pool into another (see sr_compact).
struct CompactArgs {
  const void* src;
  int64_t src_block;
  void* dst;
  int64_t dst_block;
  const int32_t* keep_flag;  // [b] or null
  const int32_t* src_row;    // [b] or null
  const int32_t* count;      // device count of kept rows (for src_row)
  int b, max_rows, n_layers, hkv, hd, elem_bytes, cap_src, cap_dst, len;
  int32_t* scratch_src_row;  // [b] used when keep_flag is given
  int32_t* new_count;        // [1] written when keep_flag is given
};
void compact(const CompactArgs& a, hipStream_t s);
// best[0] = index of the best entry of (score, cand) pairs, n >= 1.
void argmax_best(const float* score, const int32_t* cand, const int32_t* n_dev, int n_max,
                 int32_t* best, hipStream_t s);

}  // namespace sr
