// Attention of the decoder.
//
// Decode: every candidate row has one query (the newest token).  Keys are
// the prompt prefix, stored once and shared by all rows, followed by the
// row's own tail.  The query heads of one KV head are the columns of a
// v_mfma_f32_16x16x32_bf16 (S^T = K Q^T, O^T += V^T P^T), so each K/V byte is
// read once per row, and once per group of 16 / G rows for the prefix:
//   decode_group_kernel  (bf16, 64+ rows): a work-group takes a row group;
//                        its waves share the prefix blocks and split the
//                        rows' tails;
//   decode_wave_kernel   (bf16, fewer rows or no prefix): a work-group takes
//                        one (row, KV head), its waves split the keys;
//   decode_attn_kernel   (fp32 and head_dim 32): vector ALU, 16-byte loads,
//                        DPP reductions;
//   prefill_attn_mfma_kernel<.., true>: the prefix of 16 rows at once, for
//                        the one-query-head-per-KV-head case at 128+ rows.
// Online softmax in base 2; split partials are merged by log-sum-exp.
//
// Prefill (reward-model scoring, prompt): a work-group owns 8 / G blocks of
// 16 queries of one row and one KV head (MFMA flash attention, bf16
// head_dim 64/128), or a block of queries on the vector ALU with K/V staged
// in LDS as fp32.
#include <algorithm>
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace sr {

constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float exp2_or_zero(float x) { return x == -INFINITY ? 0.f : exp2f(x); }

// Work-group barrier after this wave's LDS reads and writes complete; vector
// memory loads issued before it stay in flight (__syncthreads would wait for
// them too).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// DPP move within rows of 16 lanes (ctrl: quad_perm 0x00-0xff, row_mirror
// 0x140, row_half_mirror 0x141).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

// Sum over aligned groups of LPK lanes; every lane of a group gets the sum.
// Groups of 16 use DPP within the row (xor 1, xor 2, then the mirrored
// quad and half), wider groups cross-lane shuffles.
template <int LPK>
__device__ __forceinline__ float group_sum(float d) {
  if constexpr (LPK == 16) {
    d += dpp_f32<0xB1>(d);   // quad_perm [1,0,3,2]
    d += dpp_f32<0x4E>(d);   // quad_perm [2,3,0,1]
    d += dpp_f32<0x141>(d);  // row_half_mirror
    d += dpp_f32<0x140>(d);  // row_mirror
    return d;
  } else {
#pragma unroll
    for (int o = LPK / 2; o > 0; o >>= 1) d += __shfl_xor(d, o, 64);
    return d;
  }
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

// gfx950 LDS transpose read (ds_read_b64_tr_b16).  Every lane names 8 bytes
// (four bf16); within each group of 16 lanes, element e of lane i's result
// is element (i & 3) of the four named by lane 4 e + (i >> 2).
__device__ __forceinline__ i16x4 lds_read_tr16(const bf16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p));
}
// two transpose reads as one MFMA operand (the 16-bit words reinterpreted
// as a whole vector)
__device__ __forceinline__ bf16x8 tr16_pair(i16x4 lo, i16x4 hi) {
  const i16x8 w = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, w);
}

template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
decode_attn_kernel(const float* __restrict__ q, const T* __restrict__ kpre, const T* __restrict__ vpre,
                   int P, const T* __restrict__ ktail, const T* __restrict__ vtail, int cap, int lt,
                   int hq, int hkv, int kps, int splits, float* __restrict__ part,
                   T* __restrict__ out, float qscale, int key0, int split0) {
  constexpr int EPL = Vec16<T>::N;   // elements per 16-byte load
  constexpr int LPK = HD / EPL;      // lanes per key row
  constexpr int KPW = 64 / LPK;      // keys per wave step
  constexpr int U = 4;               // keys per lane per iteration
  constexpr int NW = 4;              // waves
  // keys [key0, P + lt) in splits of kps; partial slot split0 + split
  const int split = blockIdx.x, h = blockIdx.y, row = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane % LPK, ks = lane / LPK;
  const int total = P + lt;
  const int k0 = key0 + split * kps, k1 = min(total, k0 + kps);

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

  // Raw 16-byte loads of the next U keys are issued before the current U
  // keys are consumed (two register sets, unrolled by two).
  constexpr int STEP = NW * KPW * U;
  uint4 rk0[U], rv0[U], rk1[U], rv1[U];
  auto fetch = [&](int base, uint4 (&rk)[U], uint4 (&rv)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = min(base + (u * NW + wave) * KPW + ks, k1 - 1);
      const T* kr = (j < P) ? kp + (int64_t)j * HD : kt + (int64_t)(j - P) * HD;
      const T* vr = (j < P) ? vp + (int64_t)j * HD : vt + (int64_t)(j - P) * HD;
      rk[u] = *reinterpret_cast<const uint4*>(kr + sub * EPL);
      rv[u] = *reinterpret_cast<const uint4*>(vr + sub * EPL);
    }
  };
  auto consume = [&](int base, const uint4 (&rk)[U], const uint4 (&rv)[U]) {
    float s[U][G];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = base + (u * NW + wave) * KPW + ks;
      valid[u] = j < k1;
      float kf[EPL];
      Vec16<T>::load(reinterpret_cast<const T*>(&rk[u]), kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d = fmaf(qv[g][e], kf[e], d);
        d = group_sum<LPK>(d);
        s[u][g] = valid[u] ? d : -INFINITY;
      }
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
      m[g] = mn;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[EPL];
      Vec16<T>::load(reinterpret_cast<const T*>(&rv[u]), vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = (m[g] == -INFINITY) ? 0.f : exp2_or_zero(s[u][g] - m[g]);
        l[g] += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] = fmaf(p, vf[e], acc[g][e]);
      }
    }
  };
  if (k0 < k1) {
    fetch(k0, rk0, rv0);
    for (int base = k0; base < k1; base += 2 * STEP) {
      fetch(base + STEP, rk1, rv1);
      consume(base, rk0, rv0);
      fetch(base + 2 * STEP, rk0, rv0);
      if (base + STEP < k1) consume(base + STEP, rk1, rv1);
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
    if (out) {
      out[((int64_t)row * hq + qh) * HD + dd] = from_f32<T>(A / L);
    } else {
      float* p = part + (((int64_t)row * hq + qh) * splits + split0 + split) * (HD + 2);
      p[dd] = A;
      if (dd == 0) {
        p[HD] = M;
        p[HD + 1] = L;
      }
    }
  }
}

// ------------------------------------------------ decode (waves split keys)
// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void vm_wait() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (N == 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else static_assert(N < 0, "add this wait count");
}

// 16-byte chunk slot of chunk c of key k (k = key index within a 32-key V
// block) in the LDS copy: XOR-swizzled so that the transpose reads of a
// wave (four consecutive keys per lane group, two chunks each) spread over
// the banks.
template <int CPK>
__device__ __forceinline__ int vslot(int k, int c) {
  if constexpr (CPK == 16) return c ^ (((k & 3) << 1) | (((k >> 2) & 1) << 3));
  else return c ^ ((k & 3) << 1);
}

// Decode attention over keys [key0, P + lt) for bf16, head_dim 64 or 128,
// on MFMA, with the keys split between the NW waves of a work-group (and
// between `splits` work-groups per (row, KV head)): each wave streams its
// own contiguous run of kpw keys in 32-key blocks and waits on no other wave
// until the final merge.  Work-group = (split, KV head, row); the G query
// heads of the KV head are the MFMA's 16 columns (columns >= G are zero
// queries whose results are dropped).
//   S^T = K Q^T: the A operand (16 keys x 32 dims) is loaded from memory
//         straight into registers, 16 bytes of one key row per lane.
//   O^T += V^T P^T: a V block is copied memory -> LDS (global_load_lds into
//         the wave's own double buffer) and the A operand (16 dims x 32
//         keys) comes from two LDS transpose reads; the key order of the
//         contraction is permuted so that the B operand is the lane's own 8
//         probabilities (keys 4 (l/16) + i and 16 + 4 (l/16) + i).
// The K loads and V copy of the next block are in flight while a block is
// computed.  Online softmax in base 2 (q carries log2 e / sqrt(hd)).  The
// waves' (max, sum, unnormalised output) are merged through LDS; the
// work-group writes the output or, with several splits, its partial slot.
// Fused QKV finalize (the decode step's QKV projection leaves split-K
// partials): q is summed from them and rotated here, and the wave that holds
// the newest key sums, rotates and writes its K and V row before it loads
// any key.
template <int HD, int G, int NW>
__global__ void __launch_bounds__(64 * NW)
decode_wave_kernel(const float* __restrict__ q, const bf16_t* __restrict__ kpre, const bf16_t* __restrict__ vpre,
                   int P, bf16_t* ktail, bf16_t* vtail, int cap, int lt, int hq, int hkv, int kpw, int key0,
                   int splits, float* __restrict__ part, bf16_t* __restrict__ out, float qscale,
                   const float* __restrict__ qpart, int qsplits, int qkv_dim, const float2* __restrict__ rope,
                   float* __restrict__ qout) {
  constexpr int KS = HD / 32;           // k-steps of the score product
  constexpr int DT = HD / 16;           // 16-dim tiles of the output
  constexpr int CPK = HD / 8;           // 16-byte chunks per key row
  constexpr int VB = 32 * HD;           // bf16 elements of a 32-key V block
  constexpr int NDMA = VB * 2 / 1024;   // 1 KB copies per V block
  constexpr int KPD = 64 / CPK;         // keys per copy
  constexpr int INFLIGHT = 2 * KS + NDMA;  // memory operations of one block
  static_assert(HD == 64 || HD == 128, "head_dim");
  static_assert(G >= 1 && G <= 16, "query heads per KV head");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NW * 2 * VB];
  const int split = blockIdx.x, h = blockIdx.y, row = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const int total = P + lt;
  const int w0 = key0 + (split * NW + wave) * kpw;
  const int w1 = min(total, w0 + kpw);
  const int nb = w0 < w1 ? (w1 - w0 + 31) >> 5 : 0;
  const bf16_t* kt = ktail + ((int64_t)row * hkv + h) * cap * HD;
  const bf16_t* vt = vtail + ((int64_t)row * hkv + h) * cap * HD;
  const bf16_t* kp = kpre + (int64_t)h * P * HD;
  const bf16_t* vp = vpre + (int64_t)h * P * HD;
  bf16_t* vbuf = lds + wave * 2 * VB;

  auto load_k = [&](int b, uint4 (&kr)[2][KS]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int j = min(w0 + 32 * b + 16 * t + fr, w1 - 1);
      const bf16_t* src = j < P ? kp + (int64_t)j * HD : kt + (int64_t)(j - P) * HD;
#pragma unroll
      for (int st = 0; st < KS; ++st) kr[t][st] = *reinterpret_cast<const uint4*>(src + 32 * st + 8 * fg);
    }
  };
  auto copy_v = [&](int b, int buf) {
    bf16_t* dst = vbuf + buf * VB;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const int kk = i * KPD + lane / CPK;
      const int c = vslot<CPK>(kk, lane % CPK);
      const int j = min(w0 + 32 * b + kk, w1 - 1);
      const bf16_t* src = (j < P ? vp + (int64_t)j * HD : vt + (int64_t)(j - P) * HD) + 8 * c;
      dma16(reinterpret_cast<const char*>(src), dst + i * 512);
    }
  };

  // The first block's loads go out before anything else unless it holds
  // the newest key, which this wave writes first (fused QKV finalize).
  const bool writer = qpart && nb > 0 && w1 == total;
  const bool early = nb > 0 && !(writer && nb == 1);
  uint4 ka[2][KS], kb[2][KS];
  if (early) {
    load_k(0, ka);
    copy_v(0, 0);
  }

  // fused QKV finalize: the newest key's K (rotated) and V row
  if (writer) {
    const int64_t qs = (int64_t)gridDim.z * qkv_dim;
    const float* pk = qpart + (int64_t)row * qkv_dim + (hq + h) * HD;
    const float* pv = pk + hkv * HD;
    const int64_t at = (((int64_t)row * hkv + h) * cap + lt - 1) * HD;
    for (int d = lane; d < HD / 2; d += 64) {
      float k1v = 0.f, k2v = 0.f, v1 = 0.f, v2 = 0.f;
      for (int sp = 0; sp < qsplits; ++sp) {
        k1v += pk[sp * qs + d];
        k2v += pk[sp * qs + HD / 2 + d];
        v1 += pv[sp * qs + d];
        v2 += pv[sp * qs + HD / 2 + d];
      }
      const float2 c = rope[d];
      ktail[at + d] = f32_to_bf16(k1v * c.x - k2v * c.y);
      ktail[at + HD / 2 + d] = f32_to_bf16(k2v * c.x + k1v * c.y);
      vtail[at + d] = f32_to_bf16(v1);
      vtail[at + HD / 2 + d] = f32_to_bf16(v2);
    }
    vm_wait<0>();
  }

  // Q^T fragments (B operand): lane holds Q[query fr][32 s + 8 fg .. + 8],
  // scaled, bf16.  Fused: the rotation pairs (d, d + hd/2) are the lane's
  // k-steps s and s + KS/2.
  bf16x8 qf[KS];
  {
    const bool qvalid = fr < G;
    const int qh = h * G + (qvalid ? fr : 0);
    float x[KS][8];
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int e = 0; e < 8; ++e) x[st][e] = 0.f;
    if (qpart) {
      const int64_t qs = (int64_t)gridDim.z * qkv_dim;
      const float* pq = qpart + (int64_t)row * qkv_dim + qh * HD + 8 * fg;
      if (qvalid)
        for (int sp = 0; sp < qsplits; ++sp) {
#pragma unroll
          for (int st = 0; st < KS; ++st) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(pq + sp * qs + 32 * st);
            const f32x4 b = *reinterpret_cast<const f32x4*>(pq + sp * qs + 32 * st + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x[st][e] += a[e];
              x[st][4 + e] += b[e];
            }
          }
        }
      float* qo = qout && split == 0 && wave == 0 && qvalid ? qout + ((int64_t)row * hq + qh) * HD : nullptr;
#pragma unroll
      for (int st = 0; st < KS / 2; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = 32 * st + 8 * fg + e;
          const float x1 = x[st][e], x2 = x[st + KS / 2][e];
          const float2 c = rope[d];
          x[st][e] = x1 * c.x - x2 * c.y;
          x[st + KS / 2][e] = x2 * c.x + x1 * c.y;
          if (qo) {
            qo[d] = x[st][e];
            qo[HD / 2 + d] = x[st + KS / 2][e];
          }
        }
    } else if (qvalid) {
      const float* qr = q + ((int64_t)row * hq + qh) * HD;
#pragma unroll
      for (int st = 0; st < KS; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[st][e] = qr[32 * st + 8 * fg + e];
    }
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[st][e] = (__bf16)(qvalid ? x[st][e] * qscale : 0.f);
  }

  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  // transpose-read addresses: lane names 4 dims (dt 16 + 4 (fr & 3) ..) of
  // key 4 fg + (fr >> 2), and of the key 16 on
  const int kr0 = 4 * fg + (fr >> 2), kr1 = kr0 + 16;
  auto compute = [&](int b, const uint4 (&kr)[2][KS], int buf) {
    f32x4 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2)
        st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[t][s2]), qf[s2], st[t], 0, 0,
                                                        0);
    }
    const int jb = w0 + 32 * b + 4 * fg;
    float sv[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sv[i] = jb + i < w1 ? st[0][i] : -INFINITY;
      sv[4 + i] = jb + 16 + i < w1 ? st[1][i] : -INFINITY;
    }
    float mt = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mt = fmaxf(mt, sv[i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mn = fmaxf(m, mt);
    const bool none = mn == -INFINITY;
    const float corr = none ? 1.f : exp2f(m - mn);
    bf16x8 pf;
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float pv = none ? 0.f : exp2f(sv[i] - mn);
      ps += pv;
      pf[i] = (__bf16)pv;
    }
    l = l * corr + ps;
    m = mn;
    const bf16_t* vs = vbuf + buf * VB;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int c = 2 * dt + ((fr & 3) >> 1), e4 = 4 * (fr & 1);
      const i16x4 lo = lds_read_tr16(vs + kr0 * HD + 8 * vslot<CPK>(kr0, c) + e4);
      const i16x4 hi = lds_read_tr16(vs + kr1 * HD + 8 * vslot<CPK>(kr1, c) + e4);
      o[dt] *= corr;
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tr16_pair(lo, hi), pf, o[dt], 0, 0, 0);
    }
  };

  if (nb > 0) {
    if (!early) {
      load_k(0, ka);
      copy_v(0, 0);
    }
    for (int b = 0; b < nb; b += 2) {
      if (b + 1 < nb) {
        load_k(b + 1, kb);
        copy_v(b + 1, 1);
        vm_wait<INFLIGHT>();
      } else {
        vm_wait<0>();
      }
      compute(b, ka, 0);
      if (b + 1 < nb) {
        asm volatile("" ::: "memory");
        if (b + 2 < nb) {
          load_k(b + 2, ka);
          copy_v(b + 2, 0);
          vm_wait<INFLIGHT>();
        } else {
          vm_wait<0>();
        }
        compute(b + 1, kb, 1);
        asm volatile("" ::: "memory");
      }
    }
  }

  // merge the waves: per query (max, sum, unnormalised output)
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  __syncthreads();
  float* sm = reinterpret_cast<float*>(lds);  // [NW][G][HD + 2]
  if (fr < G) {
    float* w = sm + (wave * G + fr) * (HD + 2);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) w[dt * 16 + 4 * fg + i] = o[dt][i];
    if (fg == 0) {
      w[HD] = m;
      w[HD + 1] = l;
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * HD; idx += 64 * NW) {
    const int g = idx / HD, d = idx % HD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm[(w * G + g) * (HD + 2) + HD]);
    float L = 0.f, A = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float* ws = sm + (w * G + g) * (HD + 2);
        const float c = exp2_or_zero(ws[HD] - M);
        L += ws[HD + 1] * c;
        A += ws[d] * c;
      }
    }
    const int qh = h * G + g;
    if (splits == 1 && out) {
      out[((int64_t)row * hq + qh) * HD + d] = f32_to_bf16(A / L);
    } else {
      float* pp = part + (((int64_t)row * hq + qh) * splits + split) * (HD + 2);
      pp[d] = A;
      if (d == 0) {
        pp[HD] = M;
        pp[HD + 1] = L;
      }
    }
  }
}

// Decode attention of a group of R = 16 / G rows of one KV head, the shared
// prefix attended once for the whole group (bf16, head_dim 64 or 128, MFMA).
// The 16 MFMA columns are the group's R rows x G query heads, so a prefix
// key block costs the same MFMAs as one row's tail block but serves R rows.
// Work-group = (split, KV head, row group), NW = R WPR waves: wave w takes
// an even share of the prefix blocks (all 16 columns) and one WPR-th of row
// (w mod R)'s tail blocks (the other rows' columns masked), all streamed as
// one run as in decode_wave_kernel (K into registers, V copied to the wave's
// LDS double buffer and read back transposed), with one softmax state per
// column.  The waves' partials are merged per column through LDS; the
// work-group writes the output or, with several splits, its partial slot.
// Fused QKV finalize: the wave holding a row's last tail block writes the
// row's newest K/V first.
template <int HD, int G, int WPR>
__global__ void __launch_bounds__(64 * (16 / G) * WPR)
decode_group_kernel(const float* __restrict__ q, const bf16_t* __restrict__ kpre, const bf16_t* __restrict__ vpre,
                    int P, bf16_t* ktail, bf16_t* vtail, int cap, int lt, int hq, int hkv, int rows, int splits,
                    float* __restrict__ part, bf16_t* __restrict__ out, float qscale, const float* __restrict__ qpart,
                    int qsplits, int qkv_dim, const float2* __restrict__ rope) {
  constexpr int R = 16 / G;             // rows per group
  constexpr int NW = R * WPR;           // waves
  constexpr int KS = HD / 32, DT = HD / 16, CPK = HD / 8;
  constexpr int VB = 32 * HD;
  constexpr int NDMA = VB * 2 / 1024;
  constexpr int KPD = 64 / CPK;
  constexpr int INFLIGHT = 2 * KS + NDMA;
  static_assert(HD == 64 || HD == 128, "head_dim");
  static_assert(G == 2 || G == 4 || G == 8, "query heads per KV head");
  static_assert(NW <= 8 && NW * 16 * (HD + 2) * 4 <= NW * 2 * VB * 2, "merge area within the V buffers");
  __shared__ __attribute__((aligned(1024))) bf16_t lds[NW * 2 * VB];
  const int split = blockIdx.x, h = blockIdx.y, grp = blockIdx.z;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int fr = lane & 15, fg = lane >> 4;
  const int rr = wave % R, wpart = wave / R;
  const int row = grp * R + rr;                 // this wave's tail row
  const bool rowvalid = row < rows;
  // blocks: prefix [pb0, pb1) over all splits x waves; tail [tb0, tb1) of the row
  const int nbp = (P + 31) >> 5, nbt = (lt + 31) >> 5;
  const int pi = split * NW + wave, pn = splits * NW;
  const int pb0 = nbp * pi / pn, pb1 = nbp * (pi + 1) / pn;
  const int ti = split * WPR + wpart, tn = splits * WPR;
  const int tb0 = rowvalid ? nbt * ti / tn : 0, tb1 = rowvalid ? nbt * (ti + 1) / tn : 0;
  const bf16_t* kt = ktail + ((int64_t)(rowvalid ? row : 0) * hkv + h) * cap * HD;
  const bf16_t* vt = vtail + ((int64_t)(rowvalid ? row : 0) * hkv + h) * cap * HD;
  const bf16_t* kp = kpre + (int64_t)h * P * HD;
  const bf16_t* vp = vpre + (int64_t)h * P * HD;
  bf16_t* vbuf = lds + wave * 2 * VB;

  // fused QKV finalize: the newest key's K (rotated) and V row of this row
  const bool writer = qpart && rowvalid && lt > 0 && tb1 == nbt && tb1 > tb0;
  if (writer) {
    const int64_t qs = (int64_t)rows * qkv_dim;
    const float* pk = qpart + (int64_t)row * qkv_dim + (hq + h) * HD;
    const float* pv = pk + hkv * HD;
    const int64_t at = (((int64_t)row * hkv + h) * cap + lt - 1) * HD;
    for (int d = lane; d < HD / 2; d += 64) {
      float k1v = 0.f, k2v = 0.f, v1 = 0.f, v2 = 0.f;
      for (int sp = 0; sp < qsplits; ++sp) {
        k1v += pk[sp * qs + d];
        k2v += pk[sp * qs + HD / 2 + d];
        v1 += pv[sp * qs + d];
        v2 += pv[sp * qs + HD / 2 + d];
      }
      const float2 c = rope[d];
      ktail[at + d] = f32_to_bf16(k1v * c.x - k2v * c.y);
      ktail[at + HD / 2 + d] = f32_to_bf16(k2v * c.x + k1v * c.y);
      vtail[at + d] = f32_to_bf16(v1);
      vtail[at + HD / 2 + d] = f32_to_bf16(v2);
    }
    vm_wait<0>();
  }

  // Q^T (B operand): column fr = row grp R + fr / G, query head h G + fr % G
  bf16x8 qf[KS];
  {
    const int qrow = grp * R + fr / G;
    const bool qvalid = qrow < rows;
    const int qr = qvalid ? qrow : 0, qh = h * G + fr % G;
    float x[KS][8];
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int e = 0; e < 8; ++e) x[st][e] = 0.f;
    if (qpart) {
      const int64_t qs = (int64_t)rows * qkv_dim;
      const float* pq = qpart + (int64_t)qr * qkv_dim + qh * HD + 8 * fg;
      if (qvalid)
        for (int sp = 0; sp < qsplits; ++sp) {
#pragma unroll
          for (int st = 0; st < KS; ++st) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(pq + sp * qs + 32 * st);
            const f32x4 b = *reinterpret_cast<const f32x4*>(pq + sp * qs + 32 * st + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x[st][e] += a[e];
              x[st][4 + e] += b[e];
            }
          }
        }
#pragma unroll
      for (int st = 0; st < KS / 2; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = 32 * st + 8 * fg + e;
          const float x1 = x[st][e], x2 = x[st + KS / 2][e];
          const float2 c = rope[d];
          x[st][e] = x1 * c.x - x2 * c.y;
          x[st + KS / 2][e] = x2 * c.x + x1 * c.y;
        }
    } else if (qvalid) {
      const float* qp = q + ((int64_t)qr * hq + qh) * HD;
#pragma unroll
      for (int st = 0; st < KS; ++st)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[st][e] = qp[32 * st + 8 * fg + e];
    }
#pragma unroll
    for (int st = 0; st < KS; ++st)
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[st][e] = (__bf16)(qvalid ? x[st][e] * qscale : 0.f);
  }

  // block b of a run: keys [b0 + 32 b, min(b0 + 32 b + 32, b1)) of (kb, vb)
  auto load_k = [&](const bf16_t* kb_, int k0, int k1, uint4 (&kr)[2][KS]) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int j = min(k0 + 16 * t + fr, k1 - 1);
      const bf16_t* src = kb_ + (int64_t)j * HD;
#pragma unroll
      for (int st = 0; st < KS; ++st) kr[t][st] = *reinterpret_cast<const uint4*>(src + 32 * st + 8 * fg);
    }
  };
  auto copy_v = [&](const bf16_t* vb_, int k0, int k1, int buf) {
    bf16_t* dst = vbuf + buf * VB;
#pragma unroll
    for (int i = 0; i < NDMA; ++i) {
      const int kk = i * KPD + lane / CPK;
      const int c = vslot<CPK>(kk, lane % CPK);
      const int j = min(k0 + kk, k1 - 1);
      dma16(reinterpret_cast<const char*>(vb_ + (int64_t)j * HD + 8 * c), dst + i * 512);
    }
  };
  const int kr0 = 4 * fg + (fr >> 2), kr1 = kr0 + 16;
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  // A block of a row's tail serves only that row's G columns: the other
  // columns' scores are masked, so prefix and tail blocks share one
  // softmax state per column.
  auto compute = [&](int k0, int k1, bool tail, const uint4 (&kr)[2][KS], int buf) {
    f32x4 st[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      st[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s2 = 0; s2 < KS; ++s2)
        st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[t][s2]), qf[s2], st[t], 0, 0,
                                                        0);
    }
    const int jb = k0 + 4 * fg;
    const int kend = tail && fr / G != rr ? k0 : k1;   // masked columns: no key
    float sv[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sv[i] = jb + i < kend ? st[0][i] : -INFINITY;
      sv[4 + i] = jb + 16 + i < kend ? st[1][i] : -INFINITY;
    }
    float mt = sv[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mt = fmaxf(mt, sv[i]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mn = fmaxf(m, mt);
    const bool none = mn == -INFINITY;
    const float corr = none ? 1.f : exp2f(m - mn);
    bf16x8 pf;
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float pv = none ? 0.f : exp2f(sv[i] - mn);
      ps += pv;
      pf[i] = (__bf16)pv;
    }
    l = l * corr + ps;
    m = mn;
    const bf16_t* vs = vbuf + buf * VB;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int c = 2 * dt + ((fr & 3) >> 1), e4 = 4 * (fr & 1);
      const i16x4 lo = lds_read_tr16(vs + kr0 * HD + 8 * vslot<CPK>(kr0, c) + e4);
      const i16x4 hi = lds_read_tr16(vs + kr1 * HD + 8 * vslot<CPK>(kr1, c) + e4);
      o[dt] *= corr;
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tr16_pair(lo, hi), pf, o[dt], 0, 0, 0);
    }
  };
  // The wave's blocks: its prefix share [pk0, pk1) of (kp, vp), then its
  // share [tk0, tk1) of row rr's tail in (kt, vt); one pipeline over both,
  // the next block's loads in flight while a block is computed.
  const int pk0 = 32 * pb0, pk1 = min(32 * pb1, P);
  const int tk0 = 32 * tb0, tk1 = min(32 * tb1, lt);
  const int np = pk1 > pk0 ? (pk1 - pk0 + 31) >> 5 : 0;
  const int nb = np + (tk1 > tk0 ? (tk1 - tk0 + 31) >> 5 : 0);
  auto key0 = [&](int b) { return b < np ? pk0 + 32 * b : tk0 + 32 * (b - np); };
  auto keyend = [&](int b) { return b < np ? min(pk0 + 32 * b + 32, pk1) : min(tk0 + 32 * (b - np) + 32, tk1); };
  auto fetch = [&](int b, uint4 (&kr)[2][KS], int buf) {
    const bool tail = b >= np;
    load_k(tail ? kt : kp, key0(b), keyend(b), kr);
    copy_v(tail ? vt : vp, key0(b), keyend(b), buf);
  };
  if (nb > 0) {
    uint4 ka[2][KS], kb[2][KS];
    fetch(0, ka, 0);
    for (int b = 0; b < nb; b += 2) {
      if (b + 1 < nb) {
        fetch(b + 1, kb, 1);
        vm_wait<INFLIGHT>();
      } else {
        vm_wait<0>();
      }
      compute(key0(b), keyend(b), b >= np, ka, 0);
      if (b + 1 < nb) {
        asm volatile("" ::: "memory");
        if (b + 2 < nb) {
          fetch(b + 2, ka, 0);
          vm_wait<INFLIGHT>();
        } else {
          vm_wait<0>();
        }
        compute(key0(b + 1), keyend(b + 1), b + 1 >= np, kb, 1);
        asm volatile("" ::: "memory");
      }
    }
  }

  // merge: per column c (row grp R + c / G, head h G + c % G) the partials
  // of all waves (prefix shares, and the tail shares of the row's waves)
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  __syncthreads();
  constexpr int SL = HD + 2;
  float* sp_ = reinterpret_cast<float*>(lds);   // [NW][16][SL]
  {
    float* w = sp_ + (wave * 16 + fr) * SL;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) w[dt * 16 + 4 * fg + i] = o[dt][i];
    if (fg == 0) {
      w[HD] = m;
      w[HD + 1] = l;
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 16 * HD; idx += 64 * NW) {
    const int c = idx / HD, d = idx % HD;
    const int orow = grp * R + c / G, g = c % G;
    if (orow >= rows) continue;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sp_[(w * 16 + c) * SL + HD]);
    float L = 0.f, A = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const float* ws = sp_ + (w * 16 + c) * SL;
        const float cf = exp2_or_zero(ws[HD] - M);
        L += ws[HD + 1] * cf;
        A += ws[d] * cf;
      }
    }
    const int qh = h * G + g;
    if (splits == 1) {
      out[((int64_t)orow * hq + qh) * HD + d] = f32_to_bf16(A / L);
    } else {
      float* pp = part + (((int64_t)orow * hq + qh) * splits + split) * (HD + 2);
      pp[d] = A;
      if (d == 0) {
        pp[HD] = M;
        pp[HD + 1] = L;
      }
    }
  }
}

template <typename T, int HD>
__global__ void decode_merge_kernel(const float* __restrict__ part, int splits, T* __restrict__ out) {
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

// Keys per split: aim for enough work-groups to fill the chip, at least 128
// keys per split.
static int decode_kps(int rows, int hkv, int keys) {
  int64_t groups = (int64_t)rows * hkv;
  int splits = 1;
  while (groups * splits < 2048 && keys / (splits * 2) >= 128) splits *= 2;
  return (keys + splits - 1) / splits;
}

// Waves decode_wave_kernel aims at over the whole grid.
constexpr int kWaveTarget = 2048;

template <int HD, int G, bool PREFIX_ONLY, int QB>
__global__ void prefill_attn_mfma_kernel(const float* __restrict__ q, const bf16_t* __restrict__ kpre,
                                         const bf16_t* __restrict__ vpre, int P, const bf16_t* __restrict__ kown,
                                         const bf16_t* __restrict__ vown, int rows, int lr, int cap, int t0, int hq,
                                         int hkv, bf16_t* __restrict__ out, float qscale,
                                         float* __restrict__ part, int part_splits);

// Whether the shared prefix is attended by the batched MFMA kernel (from 128
// rows; below that it costs more than the L2 reads it saves).
static bool prefix_by_mfma(int dtype, int hd, int P, int rows) {
  return dtype == SR_BF16 && hd == 128 && P > 0 && rows >= 128;
}

// Partial slots needed for `keys` = prefix + maximal tail (upper bound for
// both the combined and the split-prefix forms).
int decode_attn_splits(int rows, int hkv, int keys) {
  int kps = decode_kps(rows, hkv, keys);
  const int old_form = (keys + kps - 1) / kps + (keys + 63) / 64;
  // the key-split kernel: splits <= the waves it wants per (row, KV head),
  // which grow with the key count
  const int64_t pairs = std::max<int64_t>(1, (int64_t)rows * hkv);
  const int wave_form_max = (int)std::max<int64_t>(1, std::min<int64_t>(kWaveTarget / pairs, (keys + 31) / 32));
  return std::max(old_form, wave_form_max);
}

// Work split of decode_wave_kernel over `keys` keys of rows x hkv (row, KV
// head) pairs: about kWaveTarget waves in all (one round of resident waves:
// LDS holds ten per CU at head_dim 128), each with at least two 32-key
// blocks; NW waves per work-group (1, 2, 4 or 8) and `splits` work-groups
// per pair, each wave kpw keys (a multiple of 32).  Where eight waves per
// pair already give a thousand waves, one work-group of eight takes the pair
// (no split partials, no merge launch).
struct WavePlan {
  int nw, splits, kpw;
};
static WavePlan wave_plan(int rows, int hkv, int keys) {
  const int64_t pairs = std::max<int64_t>(1, (int64_t)rows * hkv);
  const int blocks = std::max(1, (keys + 31) / 32);
  int want = (int)std::max<int64_t>(1, kWaveTarget / pairs);
  want = std::max(1, std::min(want, blocks / 2));
  if (want > 8 && pairs * 8 >= 1024) want = 8;
  WavePlan w;
  w.nw = want >= 8 ? 8 : (want >= 4 ? 4 : (want >= 2 ? 2 : 1));
  const int per = (want + w.nw - 1) / w.nw * w.nw;    // waves per pair
  w.kpw = 32 * ((blocks + per - 1) / per);
  w.splits = std::max(1, (keys + w.nw * w.kpw - 1) / (w.nw * w.kpw));
  return w;
}

// Whether decode_wave_kernel takes these keys (bf16, head_dim 64 or 128,
// 1, 2, 4 or 8 query heads per KV head).
static bool wave_form(int dtype, int hd, int g) {
  return dtype == SR_BF16 && (hd == 64 || hd == 128) && (g == 1 || g == 2 || g == 4 || g == 8);
}

// Whether decode_group_kernel takes the launch: bf16, head_dim 64 or 128, 2,
// 4 or 8 query heads per KV head, a prefix, and from 64 rows (fewer rows
// give too few work-groups without splitting).  Waves per row: two where
// that stays within about kWaveTarget waves (not for 2 query heads per KV
// head: eight rows a group already make eight waves), else one.
constexpr int kGroupMinRows = 64;
static bool group_form(int dtype, int hd, int g, int P, int rows) {
  return dtype == SR_BF16 && (hd == 64 || hd == 128) && (g == 2 || g == 4 || g == 8) && P > 0 &&
         rows >= kGroupMinRows;
}
static int group_wpr(int g, int rows, int hkv) {
  const int R = 16 / g;
  const int64_t waves1 = (int64_t)((rows + R - 1) / R) * hkv * R;
  return (g != 2 && waves1 * 2 <= kWaveTarget + kWaveTarget / 8) ? 2 : 1;
}

template <int HD, int G>
static void launch_group(const DecodeAttnArgs& a, float qscale, hipStream_t s) {
  constexpr int R = 16 / G;
  const int wpr = group_wpr(G, a.rows, a.hkv);
  dim3 grid(1, a.hkv, (a.rows + R - 1) / R);
#define SR_GROUP(W)                                                                                               \
  SR_LAUNCH((decode_group_kernel<HD, G, W>), grid, dim3(64 * R * W), 0, s, a.q, (const bf16_t*)a.kpre,  \
                     (const bf16_t*)a.vpre, a.P, (bf16_t*)a.ktail, (bf16_t*)a.vtail, a.cap, a.lt, a.hq, a.hkv,   \
                     a.rows, 1, a.part, (bf16_t*)a.out, qscale, a.qpart, a.qsplits, a.qkv_dim, a.rope)
  if constexpr (G != 2) {
    if (wpr == 2) SR_GROUP(2);
    else SR_GROUP(1);
  } else {
    SR_GROUP(1);
  }
#undef SR_GROUP
  SR_CHECK_LAUNCH();
}

template <int HD, int G>
static void launch_wave(const DecodeAttnArgs& a, int key0, const WavePlan& w, bool direct, float qscale,
                        hipStream_t s) {
#define SR_WAVE(NW)                                                                                              \
  SR_LAUNCH((decode_wave_kernel<HD, G, NW>), dim3(w.splits, a.hkv, a.rows), dim3(64 * NW), 0, s, a.q,  \
                     (const bf16_t*)a.kpre, (const bf16_t*)a.vpre, a.P, (bf16_t*)a.ktail, (bf16_t*)a.vtail,       \
                     a.cap, a.lt, a.hq, a.hkv, w.kpw, key0, w.splits, a.part, direct ? (bf16_t*)a.out : nullptr, \
                     qscale, a.qpart, a.qsplits, a.qkv_dim, a.rope, a.qout)
  if (w.nw == 8) SR_WAVE(8);
  else if (w.nw == 4) SR_WAVE(4);
  else if (w.nw == 2) SR_WAVE(2);
  else SR_WAVE(1);
#undef SR_WAVE
  SR_CHECK_LAUNCH();
}

template <typename T, int HD, int G>
static void launch_decode(const DecodeAttnArgs& a, hipStream_t s) {
  const float qscale = kLog2e / sqrtf((float)HD);
  // The batched MFMA pass over the shared prefix (16 rows per work-group)
  // runs last: the tails leave partial slots and it folds them into its own
  // result, so no merge pass is needed.
  auto prefix_pass = [&](int tsplits) {
    SR_LAUNCH((prefill_attn_mfma_kernel<128, G, true, 1>), dim3((a.rows + 15) / 16, a.hkv, 1), dim3(64 * G), 0, s,
                       a.q, (const bf16_t*)a.kpre, (const bf16_t*)a.vpre, a.P, nullptr, nullptr, 1, a.rows, 0, 0, a.hq,
                       a.hkv, (bf16_t*)a.out, qscale, a.part, tsplits);
    SR_CHECK_LAUNCH();
  };
  if constexpr ((HD == 64 || HD == 128) && (G == 2 || G == 4 || G == 8)) {
    if (group_form(a.dtype, HD, G, a.P, a.rows)) {
      SR_REQUIRE(!a.qpart || (a.lt >= 1 && a.rope && a.qsplits >= 1), SR_ERR_INTERNAL,
                 "fused QKV finalize needs a new key");
      launch_group<HD, G>(a, qscale, s);
      return;
    }
  }
  if constexpr (HD == 64 || HD == 128) {
    if (wave_form(a.dtype, HD, G)) {
      // the key-split kernel over the keys past the prefix pass's, then the
      // prefix pass or (several splits without it) the merge
      const bool pre = prefix_by_mfma(a.dtype, HD, a.P, a.rows);
      SR_REQUIRE(!a.qpart || (a.lt >= 1 && a.rope && a.qsplits >= 1), SR_ERR_INTERNAL,
                 "fused QKV finalize needs a new key");
      const int key0 = pre ? a.P : 0;
      const int keys = a.P + a.lt - key0;
      if (keys > 0) {
        const WavePlan w = wave_plan(a.rows, a.hkv, keys);
        const bool direct = !pre && w.splits == 1;
        if (!direct)
          SR_REQUIRE((size_t)a.rows * a.hq * w.splits * (HD + 2) <= a.part_cap, 5,
                     "attention partial buffer too small");
        DecodeAttnArgs b = a;
        if (!pre) b.qout = nullptr;  // only the prefix pass reads q back
        launch_wave<HD, G>(b, key0, w, direct, qscale, s);
        if (pre) {
          prefix_pass(w.splits);
        } else if (!direct) {
          SR_LAUNCH((decode_merge_kernel<T, HD>), dim3(a.rows * a.hq), dim3(HD), 0, s, a.part, w.splits,
                             (T*)a.out);
          SR_CHECK_LAUNCH();
        }
      } else {
        prefix_pass(0);
      }
      return;
    }
  }
  SR_REQUIRE(!a.qpart, SR_ERR_INTERNAL, "fused QKV finalize without the MFMA decode kernels");
  if (prefix_by_mfma(a.dtype, HD, a.P, a.rows)) {
    // tail partials, then the prefix pass
    const int tkps = a.lt > 0 ? decode_kps(a.rows, a.hkv, a.lt) : 1;
    const int tsplits = (a.lt + tkps - 1) / tkps;
    SR_REQUIRE((size_t)a.rows * a.hq * std::max(tsplits, 1) * (HD + 2) <= a.part_cap, 5,
               "attention partial buffer too small");
    if (tsplits > 0) {
      SR_LAUNCH((decode_attn_kernel<T, HD, G>), dim3(tsplits, a.hkv, a.rows), dim3(256), 0, s, a.q,
                         (const T*)a.kpre, (const T*)a.vpre, a.P, (const T*)a.ktail, (const T*)a.vtail, a.cap,
                         a.lt, a.hq, a.hkv, tkps, tsplits, a.part, (T*)nullptr, qscale, a.P, 0);
      SR_CHECK_LAUNCH();
    }
    prefix_pass(tsplits);
    return;
  }
  const int keys = a.P + a.lt;
  const int kps = decode_kps(a.rows, a.hkv, keys);
  const int splits = (keys + kps - 1) / kps;
  if (splits > 1)
    SR_REQUIRE((size_t)a.rows * a.hq * splits * (HD + 2) <= a.part_cap, 5,
               "attention partial buffer too small");
  SR_LAUNCH((decode_attn_kernel<T, HD, G>), dim3(splits, a.hkv, a.rows), dim3(256), 0, s,
                     a.q, (const T*)a.kpre, (const T*)a.vpre, a.P, (const T*)a.ktail,
                     (const T*)a.vtail, a.cap, a.lt, a.hq, a.hkv, kps, splits, a.part,
                     splits == 1 ? (T*)a.out : (T*)nullptr, qscale, 0, 0);
  SR_CHECK_LAUNCH();
  if (splits > 1) {
    SR_LAUNCH((decode_merge_kernel<T, HD>), dim3(a.rows * a.hq), dim3(HD), 0, s, a.part,
                       splits, (T*)a.out);
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

// Whether decode_attn sums the QKV partials itself (the MFMA streaming form:
// bf16, head_dim 128, 1, 2, 4 or 8 query heads per KV head).
bool decode_attn_fuses_qkv(const DecodeAttnArgs& a) {
  if (a.hkv <= 0 || a.hq % a.hkv) return false;
  const int g = a.hq / a.hkv;
  return (g == 1 || g == 2 || g == 4 || g == 8) && a.lt >= 1 &&
         wave_form(a.dtype, a.hd, g);
}

void decode_attn(const DecodeAttnArgs& a, hipStream_t s) {
  if (a.rows <= 0) return;
  if (a.dtype == SR_BF16) decode_by_hd<bf16_t>(a, s);
  else decode_by_hd<float>(a, s);
}

// Split partials (floats) the launch of decode_attn for these arguments
// writes, following the dispatch above (without the fused QKV finalize).
size_t decode_attn_part_floats(const DecodeAttnArgs& a) {
  if (a.rows <= 0 || a.hkv <= 0 || a.hq % a.hkv) return 0;
  const int g = a.hq / a.hkv;
  const size_t per = (size_t)a.rows * a.hq * (a.hd + 2);
  if (group_form(a.dtype, a.hd, g, a.P, a.rows)) return 0;
  if (wave_form(a.dtype, a.hd, g)) {
    const bool pre = prefix_by_mfma(a.dtype, a.hd, a.P, a.rows);
    const int keys = a.P + a.lt - (pre ? a.P : 0);
    if (keys <= 0) return 0;
    const WavePlan w = wave_plan(a.rows, a.hkv, keys);
    return (!pre && w.splits == 1) ? 0 : per * w.splits;
  }
  if (prefix_by_mfma(a.dtype, a.hd, a.P, a.rows)) {
    const int tkps = a.lt > 0 ? decode_kps(a.rows, a.hkv, a.lt) : 1;
    return per * std::max((a.lt + tkps - 1) / tkps, 1);
  }
  const int keys = a.P + a.lt;
  const int kps = decode_kps(a.rows, a.hkv, keys);
  const int splits = (keys + kps - 1) / kps;
  return splits > 1 ? per * splits : 0;
}

// ---- decode attention without caller-provided scratch
// For callers that cannot allocate device memory: the split partials go to
// this file-scope array instead of a caller buffer.  Each device that runs
// the library holds its own copy until the process ends; host code reaches
// it only through the address hipGetSymbolAddress reports for the current
// device (the array's name on the host is not a device address).  Every call
// on one device shares the array, so calls that overlap on a device race.
// Every partial slot is written before it is read, so nothing is cleared.
static __device__ __align__(256) float scratch[kStaticScratchFloats];

static std::mutex g_scratch_mu;
static float* g_scratch_dev[kMaxDevices] = {};

float* static_scratch_of_current_device() {
  int dev = -1;
  SR_HIP(hipGetDevice(&dev));
  SR_REQUIRE(dev >= 0 && dev < kMaxDevices, SR_ERR_UNSUPPORTED, "device index beyond the static scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    SR_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    SR_REQUIRE(p != nullptr, SR_ERR_DEVICE, "no device address for the static scratch array");
    g_scratch_dev[dev] = static_cast<float*>(p);
  }
  return g_scratch_dev[dev];
}

// --------------------------------------------------------------- prefill
// 256 threads = QB queries x G heads x 4 threads; thread `sub` of a
// (query, head) pair owns dimensions sub, sub + 4, sub + 8, ...
template <typename T, int HD, int G>
__global__ void __launch_bounds__(256)
prefill_attn_kernel(const float* __restrict__ q, const T* __restrict__ kpre, const T* __restrict__ vpre,
                    int P, const T* __restrict__ kown, const T* __restrict__ vown, int lr, int cap, int t0,
                    int hq, int hkv, T* __restrict__ out, float qscale) {
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
  const int nkeys = P + t0 + tlast + 1;
  const T* kp = kpre + (int64_t)h * P * HD;
  const T* vp = vpre + (int64_t)h * P * HD;
  const T* ko = kown + ((int64_t)row * hkv + h) * cap * HD;
  const T* vo = vown + ((int64_t)row * hkv + h) * cap * HD;
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
      const bool ok = qvalid && key <= P + t0 + t;
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


// --------------------------------------------------------- prefill (MFMA)
// bf16 flash attention with v_mfma_f32_16x16x32_bf16, head_dim 64 or 128.
// Work-group = one row, one KV head, QB blocks of 16 queries; wave w
// computes query head (kvh * G + w % G) for query block w / G, so the G QB
// waves share every K/V tile staged in LDS.  (Two or four 16-query
// blocks per wave instead reuse a tile more but hold too many registers for
// more than one or two work-groups per SIMD, and measured slower.)
//   S^T = K Q^T   (keys x queries): lane l holds keys 4(l/16)+i (+16 for the
//                 second key tile) of query l%16, so the online-softmax state
//                 of a query lives in one lane group (max/sum over l/16).
//   O^T += V^T P^T (dims x queries): the key order of this contraction is
//                 permuted so that the B operand is exactly the lane's own
//                 S^T values (keys 4g..4g+3 of tile 0, then of tile 1); the A
//                 operand comes from the V tile, staged row by row like K, by
//                 two LDS transpose reads.
// Tiles of 64 keys (32 in the prefix pass) staged in LDS, computed 32 keys
// at a time; the next tile is fetched into registers while the current one
// is computed.
constexpr int PF_KT = 64;            // keys per staged tile (prefill form)

// PREFIX_ONLY: the decode rows' attention over the shared prompt prefix.
// The 16 "queries" of a work-group are 16 decode rows (lr = rows, one
// sequence) and every prefix key is visible.  The tails were attended first
// and left part_splits partial slots per (row, query head) in `part`
// (unnormalised output, running max, sum); the work-group folds them into
// its own result by log-sum-exp and writes the attention output.
template <int HD, int G, bool PREFIX_ONLY, int QB>
__global__ void __launch_bounds__(64 * G * QB)
prefill_attn_mfma_kernel(const float* __restrict__ q, const bf16_t* __restrict__ kpre,
                         const bf16_t* __restrict__ vpre, int P, const bf16_t* __restrict__ kown,
                         const bf16_t* __restrict__ vown, int rows, int lr, int cap, int t0, int hq, int hkv,
                         bf16_t* __restrict__ out, float qscale, float* __restrict__ part, int part_splits) {
  constexpr int NT = 64 * G * QB;
  static_assert(!PREFIX_ONLY || QB == 1, "the prefix pass takes one query block per work-group");
  // keys per staged tile: 64 for the prefill form (its work-groups have
  // eight waves to fetch them), 32 for the prefix pass (G waves)
  constexpr int KT = PREFIX_ONLY ? 32 : PF_KT;
  constexpr int KS = HD / 32, DT = HD / 16, CPK = HD / 8;
  constexpr int PF_KROW = HD + 8;    // K tile row (bf16), padded
  constexpr int PF_VROW = HD + 16;   // V tile row (bf16), padded: the 8-byte transpose reads of a
                                     // half wave (eight rows) fall on distinct banks
  static_assert(HD == 64 || HD == 128, "head_dim");
  __shared__ __attribute__((aligned(16))) bf16_t Ks[KT * PF_KROW];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[KT * PF_VROW];
  // The prefill form runs a 1-D grid of 8 C work-groups, dealt round-robin
  // to the 8 XCDs: XCD x takes the consecutive logical blocks
  // [x C, (x + 1) C), ordered query block fastest, so the query blocks that
  // read the same row's keys share one L2.
  int qb0, h, row;
  if constexpr (PREFIX_ONLY) {
    qb0 = blockIdx.x;
    h = blockIdx.y;
    row = 0;
  } else {
    const int ngq = ((lr + 15) / 16 + QB - 1) / QB, total = ngq * hkv * rows;
    const int per_xcd = (total + 7) / 8;
    const int pid = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (pid >= total) return;
    qb0 = (pid % ngq) * QB;
    h = (pid / ngq) % hkv;
    row = pid / (ngq * hkv);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  // wave w: query head h G + w % G of query block qb0 + w / G (the QB
  // blocks of a work-group share every staged K/V tile)
  const int qb = qb0 + wave / G;
  const int qh = h * G + wave % G;
  const int t = qb * 16 + fr;              // this lane's query (as B column / C column)
  const bool qvalid = t < lr;
  // Q^T fragments: lane holds Q[t][32 s + 8 fg .. +8] for k-step s (scaled,
  // bf16); loaded from a clamped row, unconditionally, so all go out at once
  bf16x8 qf[KS];
  {
    const float sc = qvalid ? qscale : 0.f;
    const float4* qr = reinterpret_cast<const float4*>(q + (((int64_t)row * lr + min(t, lr - 1)) * hq + qh) * HD);
    float4 qv[2 * KS];
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      qv[2 * st] = qr[8 * st + 2 * fg];
      qv[2 * st + 1] = qr[8 * st + 2 * fg + 1];
    }
#pragma unroll
    for (int st = 0; st < KS; ++st) {
      const float4 a = qv[2 * st], b = qv[2 * st + 1];
      qf[st][0] = (__bf16)(a.x * sc); qf[st][1] = (__bf16)(a.y * sc);
      qf[st][2] = (__bf16)(a.z * sc); qf[st][3] = (__bf16)(a.w * sc);
      qf[st][4] = (__bf16)(b.x * sc); qf[st][5] = (__bf16)(b.y * sc);
      qf[st][6] = (__bf16)(b.z * sc); qf[st][7] = (__bf16)(b.w * sc);
    }
  }
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, l = 0.f;
  // keys of the work-group's last query (its waves' masks cut the rest)
  const int tlast = min(lr, (qb0 + QB) * 16) - 1;
  const int nkeys = PREFIX_ONLY ? P : P + t0 + tlast + 1;
  const bf16_t* kp = kpre + (int64_t)h * P * HD;
  const bf16_t* vp = vpre + (int64_t)h * P * HD;
  const bf16_t* ko = PREFIX_ONLY ? kp : kown + ((int64_t)row * hkv + h) * cap * HD;
  const bf16_t* vo = PREFIX_ONLY ? vp : vown + ((int64_t)row * hkv + h) * cap * HD;
  // a tile is 32 keys x CPK chunks of 8 dims; thread chunks c = tid + NT i
  constexpr int CPT = (KT * CPK + NT - 1) / NT;
  uint4 kreg[CPT], vreg[CPT];
  auto fetch = [&](int kb) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + NT * i;
      const int key = kb + c / CPK, cc = c % CPK;
      kreg[i] = vreg[i] = make_uint4(0, 0, 0, 0);
      if (c < KT * CPK && key < nkeys) {
        const bf16_t* kr = key < P ? kp + (int64_t)key * HD : ko + (int64_t)(key - P) * HD;
        const bf16_t* vr = key < P ? vp + (int64_t)key * HD : vo + (int64_t)(key - P) * HD;
        kreg[i] = *reinterpret_cast<const uint4*>(kr + cc * 8);
        vreg[i] = *reinterpret_cast<const uint4*>(vr + cc * 8);
      }
    }
  };
  // Lane i of a group names dims dt 16 + 4 (i & 3) .. + 3 of key
  // 4 fg + (i >> 2) (and 16 keys on), so it receives dim dt 16 + i of keys
  // 4 fg .. + 3 (and 16 + 4 fg .. + 3): the A operand rows of O^T += V^T P^T
  const bf16_t* vb0 = &Vs[(4 * fg + (fr >> 2)) * PF_VROW + 4 * (fr & 3)];
  // the staged tile's keys kb .. kb + 31, at tile row r0
  auto compute = [&](int kb, int r0) {
    const bf16_t* vb = vb0 + r0 * PF_VROW;
    // S^T for key tiles 0 (keys kb..kb+15) and 1 (kb+16..kb+31)
    f32x4 st[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[(r0 + kt * 16 + fr) * PF_KROW + 32 * s + 8 * fg]);
        st[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[s], st[kt], 0, 0, 0);
      }
    }
    // causal mask and tile maximum for query t (this lane's column)
    float mt = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = kb + kt * 16 + 4 * fg + i;
        const bool ok = qvalid && key < nkeys && (PREFIX_ONLY || key <= P + t0 + t);
        st[kt][i] = ok ? st[kt][i] : -INFINITY;
        mt = fmaxf(mt, st[kt][i]);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float mn = fmaxf(m, mt);
    const float corr = (mn == -INFINITY) ? 1.f : exp2_or_zero(m - mn);
    float ls = 0.f;
    bf16x8 pf;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = (mn == -INFINITY) ? 0.f : exp2_or_zero(st[kt][i] - mn);
        ls += p;
        pf[kt * 4 + i] = (__bf16)p;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    l = l * corr + ls;
    m = mn;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      o[dt] *= corr;
      const i16x4 lo = lds_read_tr16(vb + dt * 16);
      const i16x4 hi = lds_read_tr16(vb + 16 * PF_VROW + dt * 16);
      o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(tr16_pair(lo, hi), pf, o[dt], 0, 0, 0);
    }
  };
  fetch(0);
  for (int kb = 0; kb < nkeys; kb += KT) {
    // stage K [key][dim] and V [key][dim]
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int c = threadIdx.x + NT * i;
      if (KT * CPK % NT == 0 || c < KT * CPK) {
        const int j = c / CPK, cc = c % CPK;
        *reinterpret_cast<uint4*>(&Ks[j * PF_KROW + cc * 8]) = kreg[i];
        *reinterpret_cast<uint4*>(&Vs[j * PF_VROW + cc * 8]) = vreg[i];
      }
    }
    lds_barrier();
    if (kb + KT < nkeys) fetch(kb + KT);
    compute(kb, 0);
    if (KT == 64 && kb + 32 < nkeys) compute(kb + 32, 32);
    lds_barrier();
  }
  if (qvalid) {
    if (PREFIX_ONLY) {
      // fold in the tail partials of (row t, head qh): slot s holds the
      // unnormalised output, its maximum and its sum
      const float* pr = part + ((int64_t)t * hq + qh) * part_splits * (HD + 2);
      float mx = m;
      for (int sp = 0; sp < part_splits; ++sp) mx = fmaxf(mx, pr[sp * (HD + 2) + HD]);
      const float c0 = exp2_or_zero(m - mx);
      float L = l * c0;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= c0;
      for (int sp = 0; sp < part_splits; ++sp) {
        const float* ps = pr + sp * (HD + 2);
        const float cs = exp2_or_zero(ps[HD] - mx);
        L += ps[HD + 1] * cs;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int i = 0; i < 4; ++i) o[dt][i] += ps[dt * 16 + 4 * fg + i] * cs;
      }
      const float inv = 1.0f / L;
      bf16_t* orow = out + ((int64_t)t * hq + qh) * HD;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) orow[dt * 16 + 4 * fg + i] = f32_to_bf16(o[dt][i] * inv);
    } else {
      const float inv = 1.0f / l;
      bf16_t* orow = out + (((int64_t)row * lr + t) * hq + qh) * HD;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) orow[dt * 16 + 4 * fg + i] = f32_to_bf16(o[dt][i] * inv);
    }
  }
}

template <typename T, int HD, int G>
static void launch_prefill(const PrefillAttnArgs& a, hipStream_t s) {
  constexpr int QB = 64 / G;
  const float qscale = kLog2e / sqrtf((float)HD);
  dim3 grid((a.lr + QB - 1) / QB, a.hkv, a.rows);
  SR_LAUNCH((prefill_attn_kernel<T, HD, G>), grid, dim3(256), 0, s, a.q, (const T*)a.kpre,
                     (const T*)a.vpre, a.P, (const T*)a.kown, (const T*)a.vown, a.lr, a.cap, a.t0, a.hq,
                     a.hkv, (T*)a.out, qscale);
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

// Waves per prefill work-group: G query heads x QB query blocks of 16.
constexpr int kPrefillWaves = 8;

template <int HD, int G>
static void launch_prefill_mfma(const PrefillAttnArgs& a, hipStream_t s) {
  const float qscale = kLog2e / sqrtf((float)HD);
  constexpr int QB = kPrefillWaves / G;   // query blocks per work-group
  const int64_t total = (int64_t)(((a.lr + 15) / 16 + QB - 1) / QB) * a.hkv * a.rows;
  SR_REQUIRE(total <= (int64_t)INT32_MAX - 8, SR_ERR_UNSUPPORTED, "prefill attention grid too large");
  dim3 grid((unsigned)(8 * ((total + 7) / 8)));
  SR_LAUNCH((prefill_attn_mfma_kernel<HD, G, false, QB>), grid, dim3(64 * G * QB), 0, s, a.q, (const bf16_t*)a.kpre,
                     (const bf16_t*)a.vpre, a.P, (const bf16_t*)a.kown, (const bf16_t*)a.vown, a.rows, a.lr, a.cap,
                     a.t0, a.hq, a.hkv, (bf16_t*)a.out, qscale, nullptr, 0);
  SR_CHECK_LAUNCH();
}

void prefill_attn(const PrefillAttnArgs& a, hipStream_t s) {
  if (a.rows <= 0 || a.lr <= 0) return;
  if (a.dtype == SR_BF16 && a.hd == 128) {
    switch (a.hq / a.hkv) {
      case 1: launch_prefill_mfma<128, 1>(a, s); return;
      case 2: launch_prefill_mfma<128, 2>(a, s); return;
      case 4: launch_prefill_mfma<128, 4>(a, s); return;
      case 8: launch_prefill_mfma<128, 8>(a, s); return;
      default: break;
    }
  }
  if (a.dtype == SR_BF16 && a.hd == 64) {
    switch (a.hq / a.hkv) {
      case 1: launch_prefill_mfma<64, 1>(a, s); return;
      case 2: launch_prefill_mfma<64, 2>(a, s); return;
      case 4: launch_prefill_mfma<64, 4>(a, s); return;
      case 8: launch_prefill_mfma<64, 8>(a, s); return;
      default: break;
    }
  }
  if (a.dtype == SR_BF16) prefill_by_hd<bf16_t>(a, s);
  else prefill_by_hd<float>(a, s);
}

}  // namespace sr
