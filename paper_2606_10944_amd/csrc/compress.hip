// Compress path on gfx950: v_max scan, stratified subsample and the bucketed
// kernel-halving round (KH(1/2) under kappa_att), one launch per round.
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "launch.hpp"

namespace thin {

namespace {

constexpr double kLn2 = 0.69314718055994530942;
constexpr double kLog2e = 1.44269504088896340736;

// Row strides of the index lists (0 = packed: n_r in, n_r / 2 out) and the
// first uniform of bucket t's P pairs within its slice.
__device__ __forceinline__ int64_t in_stride(const HalveArgs& a) {
  return a.in_stride ? a.in_stride : a.n_r;
}
__device__ __forceinline__ int64_t out_stride(const HalveArgs& a) {
  return a.out_stride ? a.out_stride : (a.n_r >> 1);
}
__device__ __forceinline__ int64_t bucket_u(const HalveArgs& a, int64_t t, int P) {
  return a.u_bucket ? a.u_bucket[t] : a.u_off + t * (int64_t)P;
}

__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
__device__ __forceinline__ double wave_max_d(double v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmax(v, __shfl_xor(v, off));
  return v;
}

// ---------------------------------------------------------------------------
// v_max = max_i ||v_i||_inf over the n thinned rows of a slice (Sec. 2.1, eq.
// katt); consecutive slices start slice_words 16-byte words apart.
// grid (chunks, S); the per-slice maximum is merged with an integer atomicMax
// on the float's bit pattern (valid for non-negative floats).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void vmax_kernel(const T* V, int64_t words_per_slice,
                                                   int64_t slice_words, int64_t words_per_block,
                                                   uint32_t* vmax_bits) {
  const int64_t s = blockIdx.y;
  const uint4* base = reinterpret_cast<const uint4*>(V) + s * slice_words;
  int64_t w0 = (int64_t)blockIdx.x * words_per_block;
  int64_t w1 = w0 + words_per_block;
  if (w1 > words_per_slice) w1 = words_per_slice;
  // The magnitude bits of a (non-NaN) float order like the magnitudes
  // themselves, so max |x| is taken on the bit patterns as unsigned integers
  uint32_t m = 0u;
  auto fold = [&](const u32x4& x) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (Elem<T>::bytes == 4) {
        m = max(m, x[c] & 0x7fffffffu);
      } else {
        m = max(m, (x[c] << 16) & 0x7fffffffu);
        m = max(m, x[c] & 0x7fff0000u);
      }
    }
  };
  // eight independent 16-byte loads in flight per thread
  constexpr int U = 8;
  const u32x4* vb = reinterpret_cast<const u32x4*>(base);
  int64_t w = w0 + threadIdx.x;
  for (; w + (U - 1) * (int64_t)blockDim.x < w1; w += U * (int64_t)blockDim.x) {
    u32x4 x[U];
#pragma unroll
    for (int k = 0; k < U; ++k) x[k] = vb[w + k * (int64_t)blockDim.x];
#pragma unroll
    for (int k = 0; k < U; ++k) fold(x[k]);
  }
  for (; w < w1; w += blockDim.x) fold(vb[w]);
  const float mf = wave_max_f(__uint_as_float(m));
  __shared__ float part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = mf;
  __syncthreads();
  if (threadIdx.x == 0) {
    float r = part[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = fmaxf(r, part[i]);
    atomicMax(vmax_bits + s, __float_as_uint(r));
  }
}

// p[0..count) = 0, and *also = 0 (nullable).
__global__ void zero_u32_kernel(uint32_t* p, int64_t count, int32_t* also) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0u;
  if (also && i == 0) *also = 0;
}

__global__ void zero_u8_kernel(uint8_t* p, int64_t count) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0;
}

// ---------------------------------------------------------------------------
// Stratified subsample (Alg. 3 / App. H Algorithm H.1 with unequal strata):
// stratum t = [floor(t n / n_kept), floor((t+1) n / n_kept)), pick
// start + floor(u len) computed in integers from k = floor(u 2^24).
// ---------------------------------------------------------------------------
__global__ void subsample_kernel(int64_t n, int64_t n_kept, const float* U, int64_t u_slice,
                                 int32_t* idx0) {
  const int64_t s = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_kept) return;
  const int64_t start = (t * n) / n_kept;
  const int64_t len = ((t + 1) * n) / n_kept - start;
  int64_t k = (int64_t)(U[s * u_slice + t] * 16777216.0f);
  k = k < 0 ? 0 : (k > 16777215 ? 16777215 : k);
  int64_t pick = (k * len) >> 24;
  if (pick > len - 1) pick = len - 1;
  idx0[s * n_kept + t] = (int32_t)(start + pick);
}

// dst[s, j] = src ? src[s * src_stride + j] : j   (j < n_out)
__global__ void fill_rows_kernel(int64_t n_out, const int32_t* src, int64_t src_stride,
                                 int32_t* dst) {
  const int64_t s = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n_out) return;
  dst[s * n_out + j] = src ? src[s * src_stride + j] : (int32_t)j;
}

// Output of a compress with exact sink and window rows: row j of slice s is
// sink j (j < ns), then coreset row ns + src[s * src_stride + j - ns] (src
// null = the identity) for n_out rows, then window row n - nw + ...; its
// log-weight (logw nullable) is 0 for exact rows and lw_core for coreset rows.
__global__ void assemble_kernel(int64_t n, int64_t ns, int64_t n_out, int64_t nw,
                                const int32_t* src, int64_t src_stride, int32_t* dst,
                                float* logw, float lw_core) {
  const int64_t s = blockIdx.y;
  const int64_t m = ns + n_out + nw;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  int64_t r = j;
  float w = 0.0f;
  if (j >= ns + n_out) {
    r = n - nw + (j - ns - n_out);
  } else if (j >= ns) {
    r = ns + (src ? (int64_t)src[s * src_stride + j - ns] : j - ns);
    w = lw_core;
  }
  dst[s * m + j] = (int32_t)r;
  if (logw) logw[s * m + j] = w;
}

// ---------------------------------------------------------------------------
// Cross-lane helpers (VALU only, no LDS crossbar).
// ---------------------------------------------------------------------------

// Value of lane l ^ 1 (DPP quad_perm [1,0,3,2]).
__device__ __forceinline__ uint32_t from_partner(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
}
__device__ __forceinline__ float from_partner(float v) {
  return __uint_as_float(from_partner(__float_as_uint(v)));
}
__device__ __forceinline__ double from_partner(double v) {
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint64_t r = (uint64_t)from_partner((uint32_t)u) |
                     ((uint64_t)from_partner((uint32_t)(u >> 32)) << 32);
  return __longlong_as_double((long long)r);
}

// Inclusive prefix maximum over lanes 0..31 (rows of 16 by DPP row shifts,
// then lane 15 carried into the second row).  Lanes >= 32 are ignored.
__device__ __forceinline__ double dpp_row_shr_max(double x, int n_ctrl) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint64_t ninf = (uint64_t)__double_as_longlong(-INFINITY);
  uint32_t lo, hi;
  switch (n_ctrl) {
    case 1:
      lo = __builtin_amdgcn_update_dpp((int)(uint32_t)ninf, (int)(uint32_t)u, 0x111, 0xF, 0xF, false);
      hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(ninf >> 32), (int)(uint32_t)(u >> 32), 0x111, 0xF, 0xF, false);
      break;
    case 2:
      lo = __builtin_amdgcn_update_dpp((int)(uint32_t)ninf, (int)(uint32_t)u, 0x112, 0xF, 0xF, false);
      hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(ninf >> 32), (int)(uint32_t)(u >> 32), 0x112, 0xF, 0xF, false);
      break;
    case 4:
      lo = __builtin_amdgcn_update_dpp((int)(uint32_t)ninf, (int)(uint32_t)u, 0x114, 0xF, 0xF, false);
      hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(ninf >> 32), (int)(uint32_t)(u >> 32), 0x114, 0xF, 0xF, false);
      break;
    default:
      lo = __builtin_amdgcn_update_dpp((int)(uint32_t)ninf, (int)(uint32_t)u, 0x118, 0xF, 0xF, false);
      hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(ninf >> 32), (int)(uint32_t)(u >> 32), 0x118, 0xF, 0xF, false);
      break;
  }
  return fmax(x, __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32))));
}

__device__ __forceinline__ double prefix_max32(double x, int lane) {
  x = dpp_row_shr_max(x, 1);
  x = dpp_row_shr_max(x, 2);
  x = dpp_row_shr_max(x, 4);
  x = dpp_row_shr_max(x, 8);
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint64_t r15 = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 15) |
                       ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 15) << 32);
  const double m15 = __longlong_as_double((long long)r15);
  return (lane >= 16 && lane < 32) ? fmax(x, m15) : x;
}

// exp(x) for float64 x: 2^n * 2^f with n = floor(x log2 e), 2^f from the
// float32 exp2 (about 1e-7 relative), so the range is that of float64.
__device__ __forceinline__ double exp_fast(double x) {
  const double y = x * kLog2e;
  const double n = floor(y);
  const float f = (float)(y - n);
  return ldexp((double)__builtin_amdgcn_exp2f(f), (int)n);
}

// Sum over the four lanes l, l^16, l^32, l^48 (the four column quarters of
// a row fragment); every lane receives the sum.
__device__ __forceinline__ float sum_quarters(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t w = __float_as_uint(y);
  const auto b = __builtin_amdgcn_permlane32_swap(w, w, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ double sum_quarters(double x) {
  uint64_t u = (uint64_t)__double_as_longlong(x);
  auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)u, (uint32_t)u, false, false);
  auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  double y = __longlong_as_double((long long)((uint64_t)lo[0] | ((uint64_t)hi[0] << 32))) +
             __longlong_as_double((long long)((uint64_t)lo[1] | ((uint64_t)hi[1] << 32)));
  u = (uint64_t)__double_as_longlong(y);
  lo = __builtin_amdgcn_permlane32_swap((uint32_t)u, (uint32_t)u, false, false);
  hi = __builtin_amdgcn_permlane32_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  return __longlong_as_double((long long)((uint64_t)lo[0] | ((uint64_t)hi[0] << 32))) +
         __longlong_as_double((long long)((uint64_t)lo[1] | ((uint64_t)hi[1] << 32)));
}

// ---------------------------------------------------------------------------
// Row-pair terms.  For a 16-row tile held as fragments (lane l: row l%16,
// column quarter l/16): float64 self dots <k,k>, <v,v> of every row and the
// cross dots <k,k'>, <v,v'> of every pair (rows 2q, 2q+1).  bf16: each
// v_dot2 gives two exact products summed in fp32, a partial covers 8
// elements and is accumulated in fp64; fp32: fp64 FMAs.  The cross dots use
// the partner lane's words (DPP).
// ---------------------------------------------------------------------------
// This lane's quarter of <k,k>.  Every place that forms a pair's scale h
// runs this same instruction sequence, so all of them see identical bits.
template <typename T, int D>
__device__ __forceinline__ double quarter_self_dot(const uint4* f) {
  constexpr int NW = Frag<T, D>::NV * 4;
  const uint32_t* w = reinterpret_cast<const uint32_t*>(f);
  double s = 0.0;
  if constexpr (Elem<T>::bytes == 2) {
#pragma unroll
    for (int c = 0; c < NW / 4; ++c) {
      float a = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bf16x2_t b = __builtin_bit_cast(bf16x2_t, w[4 * c + q]);
        a = __builtin_amdgcn_fdot2_f32_bf16(b, b, a, false);
      }
      s += (double)a;
    }
  } else {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const double x = (double)__uint_as_float(w[i]);
      s = fma(x, x, s);
    }
  }
  return s;
}

// This lane's quarters of <v,v>, <k,k'> and <v,v'> (k', v' = partner row).
template <typename T, int D>
__device__ __forceinline__ void quarter_pair_dots(const uint4* fk, const uint4* fv, double& sv,
                                                  double& ck, double& cv) {
  constexpr int NW = Frag<T, D>::NV * 4;
  const uint32_t* wk = reinterpret_cast<const uint32_t*>(fk);
  const uint32_t* wv = reinterpret_cast<const uint32_t*>(fv);
  sv = 0.0; ck = 0.0; cv = 0.0;
  if constexpr (Elem<T>::bytes == 2) {
#pragma unroll
    for (int c = 0; c < NW / 4; ++c) {
      float a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t xk = wk[4 * c + q], xv = wv[4 * c + q];
        const bf16x2_t bk = __builtin_bit_cast(bf16x2_t, xk);
        const bf16x2_t bv = __builtin_bit_cast(bf16x2_t, xv);
        const bf16x2_t pk = __builtin_bit_cast(bf16x2_t, from_partner(xk));
        const bf16x2_t pv = __builtin_bit_cast(bf16x2_t, from_partner(xv));
        a1 = __builtin_amdgcn_fdot2_f32_bf16(bv, bv, a1, false);
        a2 = __builtin_amdgcn_fdot2_f32_bf16(bk, pk, a2, false);
        a3 = __builtin_amdgcn_fdot2_f32_bf16(bv, pv, a3, false);
      }
      sv += (double)a1;
      ck += (double)a2;
      cv += (double)a3;
    }
  } else {
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const double xk = (double)__uint_as_float(wk[w]), xv = (double)__uint_as_float(wv[w]);
      const double pk = (double)__uint_as_float(from_partner(wk[w]));
      const double pv = (double)__uint_as_float(from_partner(wv[w]));
      sv = fma(xv, xv, sv);
      ck = fma(xk, pk, ck);
      cv = fma(xv, pv, cv);
    }
  }
}

// Scale exponent of a row: its diagonal exponent ||k||^2/sqrt(d) in base 2,
// rounded up to an integer (sk = <k,k>).  The scale of a pair is the larger
// of its two rows' values; that value is used wherever the pair's kappa
// values are scaled by 2^-h.  Integer scales keep every shifted scale
// (below) exact, and 2^(shifted - h) an exact power of two.
__device__ __forceinline__ float row_h2f(double sk, double inv_sqrt_d) {
  return (float)ceil((sk * inv_sqrt_d) * kLog2e);
}

// Extra scale of the scores of a block of rows i against pair p.  By
// Cauchy-Schwarz, <k_i,k_q>/sqrt(d) <= (e_i + e_q)/2 for the diagonal
// exponents e, so every cross exponent of a row of the block against a row q
// of pair p is at most (m_B + h_p)/2, m_B = the block's largest row scale.
// Scaling those kappa values by 2^-(h_p + shift) with
// shift = max(0, ceil((m_B - h_p)/2)) keeps every exponent <= 0 (no float32
// overflow, whatever the keys); the block's scores are then 2^-shift times
// their value at scale h_p, which the decisions undo exactly (ldexp) when
// they add the block's sums in float64.  Both arguments are integers, so
// every kernel that forms the shift gets the same value.
__device__ __forceinline__ float scale_shift(float mB, float h2) {
  return fmaxf(0.0f, ceilf(0.5f * (mB - h2)));
}
__device__ __forceinline__ float pair_h2f(float row_h2) {
  return fmaxf(row_h2, from_partner(row_h2));
}

// Row-pair terms of the 16-row tile: the row's scale exponent rh2 and its
// pair's h2f (above), and lbt = log of the RKHS distance b (Algorithm A.1)
// scaled by exp(-h/2).  The exponentials and the log are float32 (about 1e-7
// relative) on float64 arguments; the sums are float64.
template <typename T, int D>
__device__ __forceinline__ void frag_pair_terms(const uint4* fk, const uint4* fv, double vm2d,
                                                double inv_sqrt_d, float& rh2, float& h2f,
                                                float& lbt) {
  double sv, ck, cv;
  const double sk = sum_quarters(quarter_self_dot<T, D>(fk));
  quarter_pair_dots<T, D>(fk, fv, sv, ck, cv);
  sv = sum_quarters(sv);
  ck = sum_quarters(ck);
  cv = sum_quarters(cv);
  rh2 = row_h2f(sk, inv_sqrt_d);
  h2f = pair_h2f(rh2);
  const double svp = from_partner(sv);
  const double ex = sk * inv_sqrt_d, exp_ = from_partner(sk) * inv_sqrt_d, exx = ck * inv_sqrt_d;
  const double h2 = (double)h2f;
  const double t1 = (double)__builtin_amdgcn_exp2f((float)(ex * kLog2e - h2)) * (sv + vm2d);
  const double t2 = (double)__builtin_amdgcn_exp2f((float)(exp_ * kLog2e - h2)) * (svp + vm2d);
  const double t3 = (double)__builtin_amdgcn_exp2f((float)(exx * kLog2e - h2)) * (cv + vm2d);
  const double bt2 = t1 + t2 - 2.0 * t3;
  if (bt2 >= 1e-30) {
    lbt = (float)(0.5 * kLn2) * __builtin_amdgcn_logf((float)bt2);
  } else if (bt2 > 0.0) {
    // below float range: bt2 = m 2^e (hardware frexp), log2 bt2 = log2 m + e
    const float m = (float)__builtin_amdgcn_frexp_mant(bt2);
    const int e = __builtin_amdgcn_frexp_exp(bt2);
    lbt = (float)(0.5 * kLn2) * (__builtin_amdgcn_logf(m) + (float)e);
  } else {
    lbt = -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// One Halve round: KH(1/2) (App. A, Algorithm A.1) on every bucket, in two
// launches.
//
// Bucket rows y_0..y_{N-1}; pair p = (y_{2p}, y_{2p+1}).  The score of
// Algorithm A.1, alpha_p = sum_{S2} f_p - sum_{S1} f_p, is the signed sum
//     alpha_p = sum_{i<p} sgn_i E(i,p),
//     E(i,p) = k(y'_i,y_p) - k(y_i,y_p) - k(y'_i,y'_p) + k(y_i,y'_p),
// sgn_i = -1 if pair i was swapped, else +1 (the same sum, regrouped by
// earlier pair).  E does not depend on any decision, so:
//   1. pair_scores_kernel evaluates every E(i,p), i < p, of every bucket at
//      once (MFMA Gram tiles + exp), plus the per-pair terms b_i and h_i;
//   2. halve_pass_kernel takes the decisions pair by pair, in blocks of BP
//      pairs: one wavefront decides a block (ballot on alpha < a (1 - 2u),
//      the exact form of "u < min(1, (1 - alpha/a)_+ / 2)"), then every
//      wavefront adds the block's signed scores to the later pairs' alpha.
// Scaling: alpha_p is accumulated at the scale 2^h_p (h_p as in pair_h2f),
// the scale of pair p's own terms b and a; the decision only depends on
// alpha/a, which a common factor leaves unchanged.  The scores of the rows of
// one 64-row block B against p are stored at the scale 2^(h_p + shift(B,p))
// (scale_shift), which keeps every float32 exponent of the Gram epilogue at
// or below 0 whatever the keys (kappa_att overflows float32 for large keys);
// the decisions multiply each block's signed sum by 2^shift (exact) when they
// add it to alpha.  E is float32; alpha accumulates in float64.
//
// Score layout of one bucket (BR = 16 RT rows = BP pairs per block, NT =
// ceil(N/16) row tiles): panel B (the block's BP pairs as i) holds one tile
// per column tile jt = B RT .. NT-1, each tile 8 columns p x BP rows i,
// column-major ([p][i]), so a column's BP scores are contiguous.  Panel B
// starts panel_tiles(B) tiles into the bucket's array.
// ---------------------------------------------------------------------------
__host__ __device__ inline int64_t panel_tiles(int64_t B, int64_t NT, int64_t RT) {
  return B * NT - RT * B * (B - 1) / 2;
}

// Work decomposition of pair_scores_kernel.  A group is BLOCKS = W / 2
// consecutive decision blocks (64 rows each) of one bucket; each of the
// group's W waves holds one half-block (32 rows) of it as MFMA fragments
// (HB = 1 half-block per wave).  W = 8 where a half-block's fragments take at
// most four words per lane (bf16, and fp32 up to d = 64: about 128 registers
// per wave, four waves per SIMD, two workgroups per CU, whose latencies hide
// each other's), else W = 4 (fp32, d = 128).  Every launch of a bucket size
// uses the same W, so own and streamed chunks share their groups.  (Four
// waves of two half-blocks each, the two slots software-pipelined, needed
// 253 registers: two waves per SIMD, and the streamed rounds of the long
// workload ran 4-7 % slower.)  A workgroup handles one (bucket, group,
// chunk): chunk 0 covers the group's own column tiles, which the owning
// waves write to LDS from their registers (so the bucket's rows are read
// from HBM once); chunk c >= 1 covers kScoreChunk column tiles after the
// group (kScoreChunkLong in launches of many workgroups, fewer in launches of
// few), streamed from global memory through registers DEPTH tiles ahead.
#ifndef SCORE_DEPTH
#define SCORE_DEPTH 3
#endif
constexpr int kScoreStages = 3;
constexpr int kScoreChunk = 32;
constexpr int kScoreChunkLong = 48;
#ifndef SCORE_MIN_WGS
#define SCORE_MIN_WGS 128
#endif
constexpr int64_t kScoreMinWorkgroups = SCORE_MIN_WGS;  // half the CUs
constexpr int64_t kScoreLongWorkgroups = 1024;         // four per CU
// Streamed rows whose indices a workgroup stages: its chunk (at most
// kScoreChunkLong), rounded up to whole ring turns, plus the ring's
// look-ahead and the one tile whose index is read ahead of its load.
constexpr int kScoreRowsStaged = (kScoreChunkLong + 2 * SCORE_DEPTH + 2) * 16;
// A score tile (8 column pairs x 32 row pairs) in LDS: column stride 36
// floats, so the scattered single-float writes of a half-wave hit 32
// different banks.
constexpr int kETileStride = 36;
constexpr int kETileLds = 8 * kETileStride;

template <typename T, int D, int W>
struct ScoreShape {
  static constexpr int NV = Frag<T, D>::NV;
  static constexpr int HB = 1;                 // half-blocks per wave
  static constexpr int BLOCKS = W * HB / 2;    // decision blocks per group
  static constexpr int GT = 4 * BLOCKS;        // 16-row tiles per group
  static constexpr int CHUNKS = 2 * NV;        // 1 KB fragment chunks per tile (K, then V)
  static constexpr int LPT = (CHUNKS + W - 1) / W;
  // stages, score tile buffers, pair scale exponents of the group's rows,
  // row scale exponents of the stages, the half-blocks' largest row scales,
  // row indices of the streamed rows
  static constexpr int LDS = kScoreStages * CHUNKS * 1024 + kScoreStages * BLOCKS * kETileLds * 4 +
                             GT * 16 * 4 + kScoreStages * 16 * 4 + 2 * BLOCKS * 4 +
                             kScoreRowsStaged * 8;
};

// Waves of every score launch and of the local kernel (see above).
template <typename T, int D>
constexpr int score_waves() {
  return Frag<T, D>::NV < 8 ? 8 : 4;
}

// Block (group-local) and half of the half-block of wave w.
__device__ __forceinline__ void half_block(int w, int& b, int& half) {
  b = w >> 1;
  half = w & 1;
}

// The decisions of one block of 32 pairs (lane p: pair p of the block, with
// alpha = its score from earlier blocks, thr = a(1 - 2u), ef[i] = E(i, p)).
// One decision per step: the ballot of alpha < thr gives pair i's decision
// (swap: -E(i,.), else +E(i,.)), and every lane adds its signed score as one
// fused multiply-add by a uniform +-1 (the product is exact, so the result
// is the rounded sum alpha +- E).  Between the ballot and the add there are
// only scalar operations: the wave's instruction stream per decision is a
// handful of instructions, which sets this loop's speed.  No masking: lane
// p's alpha is read only at its own decision (step p), before any score of a
// pair i >= p has been added; decisions past the block's npb pairs are
// dropped.  With NEAR, en[i] = E(i, q) for a pair q of the next block, and
// near receives q's signed sum over the block (float32, in ascending i).
#ifndef DECIDE_ASM
#define DECIDE_ASM 1
#endif
template <bool NEAR>
__device__ __forceinline__ uint32_t decide_block(double alpha, double thr, const float* ef,
                                                 const float* en, int npb, float& near) {
#if DECIDE_ASM
  // One step: compare (vector, into VCC), test bit i of VCC (scalar, into
  // SCC), select +-1.0 as a float64 pair on SCC, FMA; then, off the chain,
  // the float32 +-1 for the signed sum and the decision shifted into a
  // scalar mask (decision i at bit 31 - i: mask + mask + SCC).  Four
  // instructions on the chain against five to six for the same arithmetic
  // in compiled C++, which builds the sign with shifts and masks.
  uint32_t rmask = 0;
  const double one = 1.0, mone = -1.0;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const double e = (double)ef[i];
    double sg;
    float sf;
    asm volatile(
        "v_cmp_lt_f64_e32 vcc, %[a], %[t]\n\t"
        "s_bitcmp1_b32 vcc_lo, %[i]\n\t"
        "s_cselect_b64 %[sg], %[mo], %[o]\n\t"
        "v_fmac_f64_e32 %[a], %[sg], %[e]\n\t"
        "s_cselect_b32 %[sf], -1.0, 1.0\n\t"
        "s_addc_u32 %[m], %[m], %[m]"
        : [a] "+v"(alpha), [sg] "=&s"(sg), [sf] "=&s"(sf), [m] "+s"(rmask)
        : [t] "v"(thr), [e] "v"(e), [i] "n"(i), [mo] "s"(mone), [o] "s"(one)
        : "vcc", "scc");
    if (NEAR) near = __builtin_fmaf(en[i], sf, near);
  }
  uint32_t smask = __builtin_bitreverse32(rmask);
#else
  uint32_t smask = 0;
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const double e = (double)ef[i];
    const uint32_t d = (uint32_t)(__ballot(alpha < thr) >> i) & 1u;
    smask |= d << i;
    // +-1 built as bits (the sign bit from d): scalar integer operations
    // only, no select between two vector values
    alpha = __builtin_fma(e, __hiloint2double((int)(0x3ff00000u | (d << 31)), 0), alpha);
    if (NEAR) near = __builtin_fmaf(en[i], __uint_as_float(0x3f800000u | (d << 31)), near);
  }
#endif
  if (npb < 32) smask &= (1u << npb) - 1u;
  return smask;
}

// Threshold a(1 - 2u) of the pair of lane l < 32 in a block of npb pairs
// (Algorithm A.1: a = b b_max (1/2 + log(2N/delta))), in the log domain:
// lbt = log of the pair's scaled b (-inf if b = 0), h2 = its scale exponent
// (base 2), carry = log b_max over the bucket's earlier blocks (updated to
// include this block).  a = 0 (b = 0 or b_max = 0) gives p = 1/2: swap iff
// u < 1/2.  Lanes >= 32 return values of no meaning.
__device__ __forceinline__ double block_threshold(float lbt, float h2, float u, int npb, int lane,
                                                  double log_c, double& carry) {
  const bool act = lane < npb;
  const float lbtf = act ? lbt : -INFINITY;
  const float h2f = act ? h2 : 0.0f;
  const double half_h = (double)h2f * (0.5 * kLn2);
  const double pm = prefix_max32(act ? (double)lbtf + half_h : -INFINITY, lane);
  const double lbmax = fmax(carry, pm);
  double thr;
  if (!(lbtf > -INFINITY) || !(lbmax > -INFINITY))
    thr = (u < 0.5f) ? INFINITY : -INFINITY;
  else
    thr = exp_fast((double)lbtf + lbmax + log_c - half_h) * (1.0 - 2.0 * (double)u);
  carry = __shfl(lbmax, npb - 1);
  return thr;
}

// Target of the stores of a streamed chunk's padding tiles (never read).
__device__ __align__(16) float g_score_sink[256];

// LOCAL: the whole round for buckets of at most GT*16 rows in one launch:
// one workgroup per bucket computes the bucket's scores into LDS (its own
// chunk is the whole bucket), then takes the decisions from LDS with the same
// arithmetic as halve_pass_kernel (the scores never leave the CU).
// OWN_ONLY: a launch of own chunks only (an instantiation without the
// streamed code, which needs fewer registers).
template <typename T, int D, bool LOCAL, bool OWN_ONLY, int W>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(2)))
void pair_scores_kernel(HalveArgs a) {
  using SS = ScoreShape<T, D, W>;
  constexpr int NV = SS::NV, HB = SS::HB, NBW = SS::BLOCKS, GT = SS::GT;
  constexpr int CH = SS::CHUNKS, LPT = SS::LPT;
  constexpr int BP = 32;
  constexpr int TILE = 8 * BP;
  constexpr int DEPTH = SCORE_DEPTH;
  constexpr int NS = kScoreStages;
  static_assert(DEPTH % NS == 0, "the unrolled ring keeps stage indices static");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int m16 = lane & 15;
  const int g = lane >> 4;

  const int N = a.N;
  const int P = N >> 1;
  const int NT = (N + 15) >> 4;
  const int nb = (N + 63) >> 6;
  // Workgroup -> (bucket, group, chunk).  Workgroups are dealt to the eight
  // XCDs in turn (linear id mod 8); XCD x takes buckets x, x+8, ... in sets
  // of il buckets whose workgroups are interleaved, set after set, so the
  // workgroups that share a bucket's rows share one L2 and run close
  // together.  A bucket's workgroups are its (group, chunk) pairs that have
  // work, group by group (a workgroup with nothing to do would still take a
  // dispatch slot).
  int64_t bl;
  int grp = 0, chunk = 0;
  if constexpr (LOCAL) {
    bl = blockIdx.x;
  } else {
    const int64_t id = blockIdx.x;
    const int64_t k = id >> 3;
    const int64_t per = (int64_t)a.ipb * a.il;
    const int r_ = (int)(k % per);
    bl = (id & 7) + 8 * ((k / per) * a.il + r_ % a.il);
    if (bl >= a.nbk) return;
    int item = r_ / a.il;
    for (int g_ = 0; g_ < a.ngrp; ++g_) {
      const int rest_ = NT - (g_ + 1) * GT;
      const int nsc_ = rest_ > 0 ? (rest_ + a.ch - 1) / a.ch : 0;  // streamed chunks
      const int cnt_ = max(0, min(a.chunk0 + a.nz, 1 + nsc_) - a.chunk0);
      if (item < cnt_) {
        grp = g_;
        chunk = a.chunk0 + item;
        break;
      }
      item -= cnt_;
    }
  }
  const int64_t bucket = a.b0 + bl;
  const int64_t s = bucket / a.G;
  const int64_t t = bucket % a.G;
  const int gt0 = grp * GT;  // the group's first tile
  if (gt0 >= NT) return;
  const bool own = OWN_ONLY || chunk == 0;
  const int jt0 = own ? gt0 : gt0 + GT + (chunk - 1) * a.ch;
  if (jt0 >= NT) return;
  const int jt1 = min(jt0 + (own ? GT : a.ch), NT);
  const int ntile = jt1 - jt0;

  const T* K = reinterpret_cast<const T*>(a.K) + s * a.ld * D;
  const T* V = reinterpret_cast<const T*>(a.V) + s * a.ld * D;
  const int32_t* rows_in = a.idx_in ? a.idx_in + s * in_stride(a) + t * (int64_t)N : nullptr;
  const int64_t row_base = t * (int64_t)N;
  const float vmax = __uint_as_float(a.vmax_bits[a.vmax_per_bucket ? bucket : s]);
  const float vm2f = vmax * vmax;
  const double vm2d = (double)vmax * (double)vmax;
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  const float c2 = (float)(kLog2e * inv_sqrt_d);

  extern __shared__ __align__(16) unsigned char smem[];
  // [NS][NBW] tile buffers, or (LOCAL) every score tile of the bucket
  float* s_e = reinterpret_cast<float*>(smem + NS * CH * 1024);
  float* s_h2 = s_e + (LOCAL ? (int)panel_tiles(nb, NT, 4) : NS * NBW) * kETileLds;  // [GT * 16]
  float* s_hst = s_h2 + GT * 16;                                     // [NS * 16], staged rows
  float* s_mh = s_hst + NS * 16;  // [2 * NBW]: largest row scale of each half-block
  int64_t* s_rows = reinterpret_cast<int64_t*>(s_mh + 2 * NBW);
  float* s_lbt = s_mh + 2 * NBW;  // LOCAL: pair terms [P] and [P] (no staged rows there)
  float* s_h2p = s_lbt + P;
  // LOCAL decisions: per block and lane the threshold and the bulk alpha of
  // the earlier blocks but the last ([NBW][64] each), and each block's mask
  double* s_thr = reinterpret_cast<double*>((reinterpret_cast<uintptr_t>(s_h2p + P) + 7) & ~(uintptr_t)7);
  double* s_alpha = s_thr + 64 * NBW;
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(s_alpha + 64 * NBW);

  // ---- this wave's half-blocks: fragments and, in chunk 0, pair terms ----
  int hb_blk[HB], hb_half[HB];
  bool hb_ok[HB];
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    int b, half;
    half_block(wave, b, half);
    hb_blk[h] = grp * NBW + b;
    hb_half[h] = half;
    hb_ok[h] = hb_blk[h] < nb;
  }
  // Streamed chunk: the row indices of its column rows are requested first,
  // so that their latency and the fragments' overlap (the index loads are
  // the older ones, and staging them in LDS waits for them only).
  constexpr int RPT = (kScoreRowsStaged + 64 * W - 1) / (64 * W);
  const int j_end = own ? 0 : min(N, (jt1 + 2 * DEPTH + 2) * 16);
  int64_t ridx[RPT];
  if (!own) {
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int j = jt0 * 16 + (int)threadIdx.x + k * 64 * W;
      ridx[k] = j < j_end ? (rows_in ? (int64_t)rows_in[j] : row_base + j) : 0;
    }
  }
  // This wave's rows; a streamed chunk also reads their scale exponents
  // from the per-row table (requested before the fragments, so that waiting
  // for them does not wait for the fragments).
  int64_t ar[HB][2];
  float arh[HB][2];
#pragma unroll
  for (int h = 0; h < HB; ++h)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int j = hb_blk[h] * 64 + hb_half[h] * 32 + rt * 16 + m16;
      const bool valid = hb_ok[h] && j < N;
      ar[h][rt] = valid ? (rows_in ? (int64_t)rows_in[j] : row_base + j) : -1;
      arh[h][rt] = (!own && valid) ? a.rowh2[s * a.n + ar[h][rt]] : 0.0f;
    }
  __builtin_amdgcn_sched_barrier(0);
  uint4 Ak[HB][2][NV], Av[HB][2][NV];
#pragma unroll
  for (int h = 0; h < HB; ++h)
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const bool valid = ar[h][rt] >= 0;
      const int64_t r = valid ? ar[h][rt] : 0;
      load_frag<T, D>(K, r, g, valid, Ak[h][rt]);
      load_frag<T, D>(V, r, g, valid, Av[h][rt]);
    }
  if (own) {
    // Wait for the fragments here (vmcnt(0)).  Otherwise the first use sits
    // in the tile loop, whose wait then also covers the score stores of
    // earlier tiles on every iteration (stores count in vmcnt on this
    // architecture).  Streamed chunks first use them in the peeled ring turn.
    __builtin_amdgcn_s_waitcnt(0x0F70);
    const int64_t pb = s * (a.n_r >> 1) + t * (int64_t)P;
#pragma unroll
    for (int h = 0; h < HB; ++h) {
      if (!hb_ok[h]) continue;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        float rh2, h2f, lbt;
        frag_pair_terms<T, D>(Ak[h][rt], Av[h][rt], vm2d, inv_sqrt_d, rh2, h2f, lbt);
        arh[h][rt] = ar[h][rt] >= 0 ? rh2 : 0.0f;
        const int j = hb_blk[h] * 64 + hb_half[h] * 32 + rt * 16 + m16;
        if (g == 0) s_h2[((hb_blk[h] - grp * NBW) * 4 + hb_half[h] * 2 + rt) * 16 + m16] = h2f;
        if (g == 0 && j < N && (j & 1) == 0) {
          if (LOCAL) {
            s_h2p[j >> 1] = h2f;
            s_lbt[j >> 1] = lbt;
          } else {
            a.h2[pb + (j >> 1)] = h2f;
            a.lbt[pb + (j >> 1)] = lbt;
          }
        }
        if (a.rowh2_write && g == 0 && j < N)
          a.rowh2[s * a.n + (rows_in ? (int64_t)rows_in[j] : row_base + j)] = rh2;
      }
    }
  } else {
    // row indices of every streamed column row, staged in LDS before the
    // ring starts: a data load then never waits on an index load issued
    // behind the ring's loads
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int j = jt0 * 16 + (int)threadIdx.x + k * 64 * W;
      if (j < j_end) s_rows[j - jt0 * 16] = ridx[k];
    }
  }
  // the largest row scale of each half-block (rows past the bucket: 0, and
  // every row scale is >= 0), published in LDS before the tile loop's first
  // barrier; hb_m[h] = the largest of slot h's block, read after it
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    const float mh = wave_max_f(fmaxf(arh[h][0], arh[h][1]));
    if (lane == 0) s_mh[(hb_blk[h] - grp * NBW) * 2 + hb_half[h]] = mh;
  }
  float hb_m[HB];

  // ---- column tiles ----
  // Streamed chunk c of tile jt: lane l holds row jt*16 + l%16 (clamped to
  // the bucket; rows past the end are never read back), word 4(c%NV) + l/16,
  // of K (c < NV) or V.  Own tiles are the owners' fragments, same layout.
  // Streamed rows also bring their scale exponents from the per-row table
  // (written by the first round's own chunks), staged in LDS with the rows.
  // Tiles are issued in order, and each one reads the next one's row index
  // from LDS (rnx), so that no issue waits for an LDS read.
  u32x4 stg[DEPTH][LPT];
  float hst[DEPTH];
  int64_t rnx = 0;
#define SCORE_ISSUE(JT, SLOT)                                                        \
  do {                                                                               \
    const int64_t row_ = rnx;                                                        \
    rnx = s_rows[min(((JT) + 1) * 16 + m16, N - 1) - jt0 * 16];                      \
    hst[SLOT] = a.rowh2[s * a.n + row_];                                             \
    _Pragma("unroll") for (int k_ = 0; k_ < LPT; ++k_) {                             \
      const int c_ = min(wave + k_ * W, CH - 1);                                     \
      const T* src_ = c_ < NV ? K : V;                                               \
      stg[SLOT][k_] = reinterpret_cast<const u32x4*>(src_ + row_ * D)[4 * (c_ % NV) + g]; \
    }                                                                                \
  } while (0)
#define SCORE_COMMIT(STAGE, SLOT)                                                    \
  do {                                                                               \
    if (wave == 0 && g == 0) s_hst[(STAGE) * 16 + m16] = hst[SLOT];                  \
    _Pragma("unroll") for (int k_ = 0; k_ < LPT; ++k_) {                             \
      const int c_ = wave + k_ * W;                                                  \
      if (c_ < CH) reinterpret_cast<u32x4*>(smem + ((STAGE) * CH + c_) * 1024)[lane] = stg[SLOT][k_]; \
    }                                                                                \
  } while (0)
#define SCORE_OWN_WRITE(STAGE, H, RT)                                                \
  do {                                                                               \
    _Pragma("unroll") for (int v_ = 0; v_ < NV; ++v_) {                              \
      reinterpret_cast<uint4*>(smem + ((STAGE) * CH + v_) * 1024)[lane] = Ak[H][RT][v_]; \
      reinterpret_cast<uint4*>(smem + ((STAGE) * CH + NV + v_) * 1024)[lane] = Av[H][RT][v_]; \
    }                                                                                \
  } while (0)
  // own tile TL (group-local) into a stage, by the wave holding it
#define SCORE_OWN_COMMIT(STAGE, TL)                                                  \
  do {                                                                               \
    const int b_ = (TL) >> 2, half_ = ((TL) >> 1) & 1, rt_ = (TL) & 1;              \
    if (wave == 2 * b_ + half_) {                                                    \
      if (rt_ == 0) SCORE_OWN_WRITE(STAGE, 0, 0); else SCORE_OWN_WRITE(STAGE, 0, 1);   \
    }                                                                                \
  } while (0)

  // Gram accumulators; a half-block slot h takes part in tile jt from its
  // block's diagonal on (always, in a streamed chunk).  (Two waves per SIMD
  // overlap one wave's MFMAs with the other's exp epilogue; double-buffered
  // accumulators would not fit.)
  floatx4_t gk[1][HB][2], gv[1][HB][2];
  uint4 bk_[NV], bv_[NV];
#define SCORE_ACTIVE(OWN, H, JT) (!(OWN) || (hb_ok[H] && (JT) >= hb_blk[H] * 4))
#define SCORE_BFRAG(STAGE)                                                              \
  do {                                                                                 \
    _Pragma("unroll") for (int v_ = 0; v_ < NV; ++v_) {                                \
      bk_[v_] = reinterpret_cast<const uint4*>(smem + ((STAGE) * CH + v_) * 1024)[lane]; \
      bv_[v_] = reinterpret_cast<const uint4*>(smem + ((STAGE) * CH + NV + v_) * 1024)[lane]; \
    }                                                                                  \
  } while (0)
#define SCORE_MMA_H(H)                                                                  \
  do {                                                                                 \
    _Pragma("unroll") for (int rt_ = 0; rt_ < 2; ++rt_) {                              \
      gk[0][H][rt_] = (floatx4_t){0.f, 0.f, 0.f, 0.f};                                 \
      gv[0][H][rt_] = (floatx4_t){vm2f, vm2f, vm2f, vm2f}; /* <v,v'> + v_max^2 */      \
    }                                                                                  \
    _Pragma("unroll") for (int v_ = 0; v_ < NV; ++v_)                                  \
      _Pragma("unroll") for (int rt_ = 0; rt_ < 2; ++rt_) {                            \
        gk[0][H][rt_] = mma_word<T>(Ak[H][rt_][v_], bk_[v_], gk[0][H][rt_]);           \
        gv[0][H][rt_] = mma_word<T>(Av[H][rt_][v_], bv_[v_], gv[0][H][rt_]);           \
      }                                                                                \
  } while (0)
  // Scores of slot H into the tile buffer BUF.  Lane (g, m16) holds
  // kappa(A row 4g+e, column row m16) for e = 0..3, i.e. A pairs 2g and 2g+1
  // of the row tile against column row m16.  With F = kappa(y'_i, .) -
  // kappa(y_i, .), the even lane of a column pair forms E(2g, p) =
  // F0 - F0(partner) and the odd lane E(2g+1, p) = F1(partner) - F1.
  const int epi_lane = (m16 >> 1) * kETileStride + 2 * g + (m16 & 1);
#define SCORE_EPI_H(H, H2, BUF)                                                         \
  do {                                                                                 \
    float* eb_ = LOCAL ? s_e + (panel_tiles(hb_blk[H], NT, 4) + jt_ - 4 * hb_blk[H]) * kETileLds \
                       : s_e + ((BUF) * NBW + hb_blk[H] - grp * NBW) * kETileLds;      \
    const float he_ = (H2) + scale_shift(hb_m[H], (H2));                               \
    _Pragma("unroll") for (int rt = 0; rt < 2; ++rt) {                                 \
      float kap[4];                                                                    \
      _Pragma("unroll") for (int e = 0; e < 4; ++e)                                    \
        kap[e] = __builtin_amdgcn_exp2f(gk[0][H][rt][e] * c2 - he_) * gv[0][H][rt][e]; \
      const float F0 = kap[1] - kap[0];                                                \
      const float F1 = kap[3] - kap[2];                                                \
      const float mine_ = odd ? F1 : F0;                                               \
      const float other_ = from_partner(odd ? F0 : F1);                                \
      eb_[epi_lane + hb_half[H] * 16 + rt * 8] =                                       \
          odd ? other_ - mine_ : mine_ - other_;                                       \
    }                                                                                  \
  } while (0)
  // Wave w < NBW writes block w's completed tile IF (buffer BUF) to the score
  // array: 16 bytes per lane, 128 contiguous bytes per column pair.  A
  // streamed chunk's padding tiles go to the sink.
#define SCORE_FLUSH(OWN, IF, BUF)                                                       \
  do {                                                                                 \
    if (!LOCAL && (NBW == W || wave < NBW)) {                                          \
      const int bw_ = grp * NBW + wave;                                                \
      const int jtf_ = jt0 + (IF);                                                     \
      if (!(OWN) || (bw_ < nb && jtf_ >= 4 * bw_)) {                                   \
        float* dst_ = (OWN) || (IF) < ntile                                            \
            ? a.E + (bl * a.e_tiles + panel_tiles(bw_, NT, 4) + jtf_ - 4 * bw_) * (int64_t)TILE \
            : g_score_sink;                                                            \
        const float4 v_ = *reinterpret_cast<const float4*>(                            \
            s_e + ((BUF) * NBW + wave) * kETileLds + (lane >> 3) * kETileStride + (lane & 7) * 4); \
        *reinterpret_cast<float4*>(dst_ + (lane >> 3) * BP + (lane & 7) * 4) = v_;     \
      }                                                                                \
    }                                                                                  \
  } while (0)
  // Streamed tiles: the column fragments are read from the stage word by
  // word beside the MFMAs that use them (all of them at once would take 32
  // more registers, past the 128 that four waves per SIMD allow)
#define SCORE_MMA_LDS(H, STAGE)                                                         \
  do {                                                                                 \
    _Pragma("unroll") for (int rt_ = 0; rt_ < 2; ++rt_) {                              \
      gk[0][H][rt_] = (floatx4_t){0.f, 0.f, 0.f, 0.f};                                 \
      gv[0][H][rt_] = (floatx4_t){vm2f, vm2f, vm2f, vm2f};                             \
    }                                                                                  \
    _Pragma("unroll") for (int v_ = 0; v_ < NV; ++v_) {                                \
      const uint4 bk1_ = reinterpret_cast<const uint4*>(smem + ((STAGE) * CH + v_) * 1024)[lane]; \
      const uint4 bv1_ = reinterpret_cast<const uint4*>(smem + ((STAGE) * CH + NV + v_) * 1024)[lane]; \
      _Pragma("unroll") for (int rt_ = 0; rt_ < 2; ++rt_) {                            \
        gk[0][H][rt_] = mma_word<T>(Ak[H][rt_][v_], bk1_, gk[0][H][rt_]);              \
        gv[0][H][rt_] = mma_word<T>(Av[H][rt_][v_], bv1_, gv[0][H][rt_]);              \
      }                                                                                \
    }                                                                                  \
  } while (0)

  // One column tile (tile I of the chunk, ring position U = I mod 3): tile
  // I+2 staged (and, streamed, tile I+2+DEPTH loaded), Grams and scores of
  // tile I, then the previous tile written out (its LDS read after this
  // tile's work, so that it waits at the barrier's wait only).
#define SCORE_TILE(OWN, I, U)                                                           \
  do {                                                                                 \
    const int i_ = (I);                                                                \
    const int jt_ = jt0 + i_;                                                          \
    if (OWN) {                                                                         \
      if (i_ + 2 < ntile) SCORE_OWN_COMMIT(((U) + 2) % NS, i_ + 2);                    \
    } else {                                                                           \
      SCORE_COMMIT(((U) + 2) % NS, ((U) + 2) % DEPTH);                                 \
      SCORE_ISSUE(jt_ + 2 + DEPTH, ((U) + 2) % DEPTH);                                 \
    }                                                                                  \
    if (OWN) SCORE_BFRAG((U) % NS);                                                    \
    const float h2_ = jt_ * 16 + m16 >= N ? 0.0f                                       \
                      : (OWN) ? s_h2[i_ * 16 + m16] : pair_h2f(s_hst[((U) % NS) * 16 + m16]);        \
    _Pragma("unroll") for (int h = 0; h < HB; ++h) {                                   \
      if (!SCORE_ACTIVE(OWN, h, jt_)) continue;                                        \
      if (OWN) SCORE_MMA_H(h); else SCORE_MMA_LDS(h, (U) % NS);                        \
      SCORE_EPI_H(h, h2_, (U) % NS);                                                   \
    }                                                                                  \
    if (i_ > 0) SCORE_FLUSH(OWN, i_ - 1, ((U) + NS - 1) % NS);                         \
    __syncthreads();                                                                   \
  } while (0)
  // LOCAL: the decisions of the bucket's P <= 32 NBW pairs from the scores
  // in LDS, with the arithmetic of halve_pass_kernel: block m's thresholds,
  // then alpha = the float32 signed sums of every earlier block added in
  // block order in float64, then decide_block.  Every wave of the workgroup
  // takes part.  First wave m < nblk forms block m's thresholds (the carry
  // of the earlier blocks is the largest of their pairs' values, which the
  // sequential scan carries forward).  Then block by block, one barrier
  // each: wave 0 adds the previous block's sums to the alpha the helpers
  // have built and decides the block; meanwhile waves 1.. add that previous
  // block's sums to the alpha of the blocks after this one, in block order,
  // so every alpha is the same float64 sum as one wave's.
  auto local_decisions = [&]() {
    const int nblk = (P + 31) / 32;
    const float* Ub = a.U + s * a.u_slice + bucket_u(a, t, P);
    uint8_t* trace = a.trace ? a.trace + s * a.u_slice + bucket_u(a, t, P) : nullptr;
    int32_t* out = a.idx_out + s * out_stride(a) + t * (int64_t)P;
    const int pl = lane & 31;
    auto pair_of = [&](int m) { return 32 * m + min(pl, min(32, P - 32 * m) - 1); };
    // block b's signed sums at pair gp's scale (gp in a later block)
    auto bulk = [&](int b, uint32_t mask, int gp) {
      const float* col = s_e + (panel_tiles(b, NT, 4) + (gp >> 3) - 4 * b) * kETileLds + (gp & 7) * kETileStride;
      float sum = 0.0f;
#pragma unroll
      for (int i = 0; i < 32; ++i) sum += ((mask >> i) & 1u) ? -col[i] : col[i];
      return ldexp((double)sum, (int)scale_shift(fmaxf(s_mh[2 * b], s_mh[2 * b + 1]), s_h2p[gp]));
    };
    if (wave < nblk) {
      const int m = wave;
      const int npb = min(32, P - 32 * m);
      const int gp = pair_of(m);
      double carry = -INFINITY;
      for (int b = 0; b < m; ++b) {  // earlier blocks are whole
        const int q = 32 * b + pl;
        carry = fmax(carry, (double)s_lbt[q] + (double)s_h2p[q] * (0.5 * kLn2));
      }
      carry = wave_max_d(carry);
      s_thr[64 * m + lane] = block_threshold(s_lbt[gp], s_h2p[gp], Ub[gp], npb, lane, a.log_c, carry);
    }
    for (int k = threadIdx.x; k < 64 * NBW; k += 64 * W) s_alpha[k] = 0.0;
    __syncthreads();
    uint32_t prev = 0u;  // wave 0: the last block's mask
    for (int m = 0; m < nblk; ++m) {
      if (wave == 0) {
        const int npb = min(32, P - 32 * m);
        const int gp = pair_of(m);
        double alpha = s_alpha[64 * m + lane];
        if (m > 0) alpha += bulk(m - 1, prev, gp);
        float ef[32];
        const float* oc = s_e + (panel_tiles(m, NT, 4) + (gp >> 3) - 4 * m) * kETileLds + (gp & 7) * kETileStride;
#pragma unroll
        for (int i = 0; i < 32; ++i) ef[i] = oc[i];
        float unused = 0.0f;
        // the block's own scores are at its shifted scale: decide there
        const int sh = (int)scale_shift(fmaxf(s_mh[2 * m], s_mh[2 * m + 1]), s_h2p[gp]);
        prev = decide_block<false>(ldexp(alpha, -sh), ldexp(s_thr[64 * m + lane], -sh), ef, ef, npb,
                                   unused);
        if (lane == 0) s_mask[m] = prev;
        const uint32_t bit = (prev >> pl) & 1u;
        if (lane < npb) {
          const int32_t r0 = rows_in ? rows_in[2 * gp] : (int32_t)(row_base + 2 * gp);
          const int32_t r1 = rows_in ? rows_in[2 * gp + 1] : (int32_t)(row_base + 2 * gp + 1);
          out[gp] = bit ? r1 : r0;
          if (trace) trace[gp] = (uint8_t)bit;
        }
      } else if (m > 0 && m + wave < nblk) {
        const int j = m + wave;  // a later block: block m - 1's sums join its alpha
        s_alpha[64 * j + lane] += bulk(m - 1, s_mask[m - 1], pair_of(j));
      }
      __syncthreads();
    }
  };

  const bool odd = (m16 & 1) != 0;
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HB; ++h) {
    const int lb = hb_blk[h] - grp * NBW;
    hb_m[h] = fmaxf(s_mh[2 * lb], s_mh[2 * lb + 1]);
  }
  // the decision pass reads each block's largest row scale from here
  if (!LOCAL && own && (int)threadIdx.x < NBW && grp * NBW + (int)threadIdx.x < nb)
    a.mB[bucket * nb + grp * NBW + threadIdx.x] =
        fmaxf(s_mh[2 * threadIdx.x], s_mh[2 * threadIdx.x + 1]);
  if (own) {
    SCORE_OWN_COMMIT(0, 0);
    if (ntile > 1) SCORE_OWN_COMMIT(1, 1);
    __syncthreads();
    for (int ib = 0; ib < ntile; ib += DEPTH) {
#pragma unroll
      for (int u = 0; u < DEPTH; ++u)
        if (ib + u < ntile) SCORE_TILE(true, ib + u, u);  // uniform over the workgroup
    }
    SCORE_FLUSH(true, ntile - 1, (ntile - 1) % NS);
    if constexpr (LOCAL) {
      __syncthreads();
      local_decisions();
    }
  } else if constexpr (!LOCAL && !OWN_ONLY) {
    rnx = s_rows[min(jt0 * 16 + m16, N - 1) - jt0 * 16];  // staged before the barrier above
#pragma unroll
    for (int k = 0; k < DEPTH; ++k) SCORE_ISSUE(jt0 + k, k);
    SCORE_COMMIT(0, 0);
    SCORE_COMMIT(1, 1);
    SCORE_ISSUE(jt0 + DEPTH, 0);
    SCORE_ISSUE(jt0 + DEPTH + 1, 1);
    __syncthreads();
    // The first ring turn is peeled: the loop is then entered with the same
    // loads and stores in flight as at its back edge, so the compiler's wait
    // for a staged tile is for that tile's loads only, not for the stores
    // issued after them (stores count in vmcnt on this architecture).  The
    // chunk runs whole ring turns (tiles past ntile are padding).
    const int nturn = (ntile + DEPTH - 1) / DEPTH;
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) SCORE_TILE(false, u, u);
    for (int ib = DEPTH; ib < nturn * DEPTH; ib += DEPTH) {
#pragma unroll
      for (int u = 0; u < DEPTH; ++u) SCORE_TILE(false, ib + u, u);
    }
    SCORE_FLUSH(false, nturn * DEPTH - 1, (nturn * DEPTH - 1) % NS);
  }
#undef SCORE_TILE
#undef SCORE_MMA_LDS
#undef SCORE_FLUSH
#undef SCORE_EPI_H
#undef SCORE_MMA_H
#undef SCORE_BFRAG
#undef SCORE_ACTIVE
#undef SCORE_ISSUE
#undef SCORE_COMMIT
#undef SCORE_OWN_WRITE
#undef SCORE_OWN_COMMIT
}

// Buckets of at most 64 rows (one decision block of P <= 32 pairs): one
// wavefront per bucket, eight buckets per workgroup, the whole round in
// registers and a 4 KiB score tile in LDS.  The arithmetic is the local
// kernel's, step for step (the same Gram words in the same order, the same
// epilogue, scales, thresholds and decision loop), so both take the same
// decisions; what changes is the size of the work unit: the local kernel
// gives a whole workgroup of eight waves to a bucket, which at 16-64 rows
// leaves most of them idle (the prefill's Compress2 calls are 16-row buckets,
// 98304 of them in one launch).  RT = 16-row tiles per bucket (N <= 16 RT).
constexpr int kTinyWaves = 8;
#ifndef TINY_MIN_BUCKETS
#define TINY_MIN_BUCKETS 1024
#endif
constexpr int64_t kTinyMinBuckets = TINY_MIN_BUCKETS;  // launches with fewer take the local kernel
constexpr int kTinyStride = 33;  // floats per score row in LDS (rows i, columns p)

template <typename T, int D, int RT>
__global__ __launch_bounds__(64 * kTinyWaves) void tiny_halve_kernel(HalveArgs a) {
  constexpr int NV = Frag<T, D>::NV;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const bool odd = (m16 & 1) != 0;
  const int64_t bl = (int64_t)blockIdx.x * kTinyWaves + wave;
  if (bl >= a.nbk) return;  // no barrier below: a wave without a bucket just ends
  const int N = a.N, P = N >> 1;
  const int64_t bucket = a.b0 + bl;
  const int64_t s = bucket / a.G, t = bucket % a.G;
  const T* K = reinterpret_cast<const T*>(a.K) + s * a.ld * D;
  const T* V = reinterpret_cast<const T*>(a.V) + s * a.ld * D;
  const int32_t* rows_in = a.idx_in ? a.idx_in + s * in_stride(a) + t * (int64_t)N : nullptr;
  const int64_t row_base = t * (int64_t)N;
  const float vmax = __uint_as_float(a.vmax_bits[a.vmax_per_bucket ? bucket : s]);
  const float vm2f = vmax * vmax;
  const double vm2d = (double)vmax * (double)vmax;
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  const float c2 = (float)(kLog2e * inv_sqrt_d);

  __shared__ float s_e[kTinyWaves][32 * kTinyStride];  // E(i, p) at [i * stride + p]
  __shared__ float s_h2p[kTinyWaves][32], s_lbt[kTinyWaves][32];
  float* e = s_e[wave];

  // rows and their fragments
  int64_t ar[RT];
  uint4 Ak[RT][NV], Av[RT][NV];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int j = rt * 16 + m16;
    ar[rt] = j < N ? (rows_in ? (int64_t)rows_in[j] : row_base + j) : -1;
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const bool valid = ar[rt] >= 0;
    load_frag<T, D>(K, valid ? ar[rt] : 0, g, valid, Ak[rt]);
    load_frag<T, D>(V, valid ? ar[rt] : 0, g, valid, Av[rt]);
  }
  // pair terms; the block's largest row scale (rows past the bucket: 0)
  float h2c[RT];
  float mB = 0.0f;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    float rh2, h2f, lbt;
    frag_pair_terms<T, D>(Ak[rt], Av[rt], vm2d, inv_sqrt_d, rh2, h2f, lbt);
    const int j = rt * 16 + m16;
    h2c[rt] = j < N ? h2f : 0.0f;
    mB = fmaxf(mB, ar[rt] >= 0 ? rh2 : 0.0f);
    if (g == 0 && j < N && (j & 1) == 0) {
      s_h2p[wave][j >> 1] = h2f;
      s_lbt[wave][j >> 1] = lbt;
    }
    if (a.rowh2_write && g == 0 && j < N) a.rowh2[s * a.n + ar[rt]] = rh2;
  }
  mB = wave_max_f(mB);
  // scores of every row tile against every column tile from its diagonal on
#pragma unroll
  for (int ct = 0; ct < RT; ++ct) {
    const float he = h2c[ct] + scale_shift(mB, h2c[ct]);
#pragma unroll
    for (int rt = 0; rt <= ct; ++rt) {
      floatx4_t gk = {0.f, 0.f, 0.f, 0.f};
      floatx4_t gv = {vm2f, vm2f, vm2f, vm2f};  // <v,v'> + v_max^2
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        gk = mma_word<T>(Ak[rt][v], Ak[ct][v], gk);
        gv = mma_word<T>(Av[rt][v], Av[ct][v], gv);
      }
      float kap[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) kap[q] = __builtin_amdgcn_exp2f(gk[q] * c2 - he) * gv[q];
      const float F0 = kap[1] - kap[0];
      const float F1 = kap[3] - kap[2];
      const float mine = odd ? F1 : F0;
      const float other = from_partner(odd ? F0 : F1);
      // lane (g, m16): pair i = 8 rt + 2 g + odd of the row tile against pair
      // p = 8 ct + m16 / 2 of the column tile
      e[(8 * rt + 2 * g + (odd ? 1 : 0)) * kTinyStride + 8 * ct + (m16 >> 1)] =
          odd ? other - mine : mine - other;
    }
  }
  // the wave's score writes are complete before any lane reads another's
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // the block's decisions (no earlier block: alpha starts at zero)
  const int pl = lane & 31;
  const int gp = min(pl, P - 1);
  const float* Ub = a.U + s * a.u_slice + bucket_u(a, t, P);
  double carry = -INFINITY;
  const double thr = block_threshold(s_lbt[wave][gp], s_h2p[wave][gp], Ub[gp], P, lane, a.log_c,
                                     carry);
  const int sh = (int)scale_shift(mB, s_h2p[wave][gp]);
  float ef[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) ef[i] = e[i * kTinyStride + gp];
  float unused = 0.0f;
  const uint32_t smask = decide_block<false>(ldexp(0.0, -sh), ldexp(thr, -sh), ef, ef, P, unused);
  if (lane < P) {
    const uint32_t bit = (smask >> pl) & 1u;
    const int32_t r0 = rows_in ? rows_in[2 * gp] : (int32_t)(row_base + 2 * gp);
    const int32_t r1 = rows_in ? rows_in[2 * gp + 1] : (int32_t)(row_base + 2 * gp + 1);
    a.idx_out[s * out_stride(a) + t * (int64_t)P + gp] = bit ? r1 : r0;
    if (a.trace) a.trace[s * a.u_slice + bucket_u(a, t, P) + gp] = (uint8_t)bit;
  }
}

// Decision pass of one bucket per workgroup, in three roles that run ahead
// of or behind each other, synchronised by progress counters in LDS:
//  - wave 1 (fetcher) stages each block's inputs in a ring of FD + 1 LDS
//    slots, up to FD blocks ahead of the decider (FD blocks' loads in flight):
//    the block's own scores, the scores
//    against the next block's pairs, the row indices, and the thresholds
//    a(1 - 2u), which depend on no decision (the running maximum of b over
//    the bucket is carried from block to block);
//  - wave 0 (decider) takes the decisions of a block two at a time (the
//    second decision is evaluated for both outcomes of the first), publishes
//    them, then adds the block's scores to the next block's pairs itself;
//  - waves 2.. (bulk) add each decided block's scores to all pairs two or
//    more blocks later.  Each pair belongs to one bulk wave (64-pair chunks,
//    dealt round robin), which adds the blocks in order; the column chunks
//    are fetched ahead in one stream per wave, across blocks.
// alpha of a pair in block m = (contributions of blocks <= m-2, summed by the
// bulk waves in block order) + (contribution of block m-1, from the decider).
// The decider never waits on global memory.  Every wait is bounded.
constexpr int kSpinLimit = 1 << 16;

// Returns the last value read (>= target unless the spin limit ran out).  A
// wait that runs out sets the call's status word (status nullable): the
// kernel still ends normally, and the caller learns that this call's
// decisions cannot be trusted.
__device__ __forceinline__ int wait_at_least(const int* flag, int target, int32_t* status) {
  int v = 0;
  for (int it = 0; it < kSpinLimit; ++it) {
    v = __hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
    if (v >= target) return v;
    __builtin_amdgcn_s_sleep(1);
  }
  if (status) __hip_atomic_store(status, kStatusWaitExhausted, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return v;
}
__device__ __forceinline__ void publish(int* flag, int value) {
  __hip_atomic_store(flag, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Decision helpers: rows 0 .. hand_row(c) of chunk c are added by helper
// workgroups, the last kPassHand rows before the chunk's first block by the
// bucket's own bulk waves (the hand-over then has kPassHand + 1 blocks of
// decisions to arrive before the decider needs the chunk).
#ifndef PASS_HAND
#define PASS_HAND 10
#endif
constexpr int kPassHand = PASS_HAND;
__device__ __forceinline__ int hand_row(int c) { return 2 * c - 2 - kPassHand; }
// Every access to the words the helpers share with the bucket's workgroup
// (decisions, flags, partials) is a read-modify-write atomic at agent scope:
// all of them are then performed at one place, the L2 of the XCD that runs
// the bucket's workgroup and its helpers (pass_helpers keeps them on one),
// so a flag seen there covers the partials written before it.
// The word reads and the flag updates are made once per wave (lane 0, the
// result broadcast): lanes that each update one flag would each see another
// old value.
__device__ __forceinline__ uint64_t shared_read(uint64_t* p) {
  uint64_t v = 0;
  if ((threadIdx.x & 63) == 0) v = __hip_atomic_fetch_add(p, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __shfl(v, 0);
}
__device__ __forceinline__ uint32_t shared_read(uint32_t* p) {
  uint32_t v = 0;
  if ((threadIdx.x & 63) == 0) v = __hip_atomic_fetch_add(p, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __shfl(v, 0);
}
// flag = max(flag, v); returns the old value (wave-uniform)
__device__ __forceinline__ uint32_t shared_max(uint32_t* p, uint32_t v) {
  uint32_t old = 0;
  if ((threadIdx.x & 63) == 0) old = __hip_atomic_fetch_max(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return __shfl(old, 0);
}
// per lane (each lane its own word)
__device__ __forceinline__ uint64_t shared_read_lane(uint64_t* p) {
  return __hip_atomic_fetch_add(p, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void shared_write(uint64_t* p, uint64_t v) {
  (void)__hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Tag of block m's decisions in a round: nonzero, distinct per round and block.
__device__ __forceinline__ uint32_t helper_tag(int32_t round_tag, int m) {
  return ((uint32_t)round_tag << 16) | (uint32_t)(m + 1);
}
// The decisions in a tagged word once its tag is `tag` (`w` read ahead;
// bounded wait at agent scope, like wait_at_least).
__device__ __forceinline__ uint32_t decided_mask(uint64_t* p, uint64_t w, uint32_t tag,
                                                 int32_t* status) {
  for (int it = 0; (uint32_t)(w >> 32) != tag; ++it) {
    if (it == kSpinLimit) {
      if (status) __hip_atomic_store(status, kStatusWaitExhausted, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
    w = shared_read(p);
  }
  return (uint32_t)w;
}
__device__ __forceinline__ void wait_flag(uint32_t* p, uint32_t value, int32_t* status) {
  uint32_t v = shared_read(p);
  for (int it = 0; v < value; ++it) {
    if (it == kSpinLimit) {
      if (status) __hip_atomic_store(status, kStatusWaitExhausted, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
    v = shared_read(p);
  }
}

template <int BW, int NCB, int FD>
struct PassLds {
  static constexpr int BP = 32, QW = 8, NSLOT = FD + 1;
  // alpha [P] f64 | decisions of every block [nblk] u32 | counters [16]:
  // last decided block, last staged block, rows completed by each bulk wave |
  // NSLOT input slots, each: thresholds [BP] f64, rows [2][BP] i32, own
  // scores [BP][CW] and next-block scores [BP][CW] 16-byte words | with
  // COAL, per bulk wave a column buffer [64][CW] 16-byte words.  A column of
  // BP scores is QW words plus one of padding (CW): reads of whole columns
  // by consecutive lanes then fall in different banks.  COAL: the bulk waves
  // load their chunks coalesced and transpose them in LDS (with six bulk
  // waves, on the largest buckets, the loads limit the bulk); else each lane
  // loads its own column: less LDS, and the decider's LDS accesses do not
  // queue behind the transposes.
  static constexpr int CW = QW + 1;
  static constexpr bool COAL = BW >= 6;
  static constexpr size_t kSlot = BP * 8 + 2 * BP * 4 + 2 * BP * CW * 16;
  static constexpr size_t kColBuf = COAL ? 64 * CW * 16 : 0;
  static_assert(2 + BW <= 16, "counter block");
  __host__ __device__ static size_t mask_off(int P) { return ((size_t)P * 8 + 15) & ~(size_t)15; }
  __host__ __device__ static size_t flag_off(int P) {
    return mask_off(P) + (((size_t)(P + BP - 1) / BP * 4 + 15) & ~(size_t)15);
  }
  __host__ __device__ static size_t slot_off(int P) { return flag_off(P) + 64; }
  __host__ __device__ static size_t colbuf_off(int P) { return slot_off(P) + NSLOT * kSlot; }
  // pair scale exponents [P] f32 | largest row scale of every block [nblk] f32
  __host__ __device__ static size_t h2_off(int P) { return colbuf_off(P) + BW * kColBuf; }
  __host__ __device__ static size_t mb_off(int P) { return h2_off(P) + (((size_t)P * 4 + 15) & ~(size_t)15); }
  // rows of bulk sums completed per 64-pair chunk [nch] i32
  __host__ __device__ static size_t chunk_off(int P) {
    return mb_off(P) + (((size_t)(P + BP - 1) / BP * 4 + 15) & ~(size_t)15);
  }
  __host__ __device__ static size_t bytes(int P) {
    return chunk_off(P) + (((size_t)(P + 63) / 64 * 4 + 15) & ~(size_t)15);
  }
};

template <int BW, int NCB, int FD, bool HELP>
__global__ __launch_bounds__(64 * (BW + 2)) void halve_pass_kernel(HalveArgs a) {
  using L = PassLds<BW, NCB, FD>;
  constexpr int RT = 4;
  constexpr int BR = 16 * RT;
  constexpr int BP = BR / 2;
  constexpr int TILE = 8 * BP;
  constexpr int QW = BP / 4;  // 16-byte words per score column
  static_assert(BP == L::BP && QW == L::QW, "layout");

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // with helpers: workgroups [0, nbk) take their bucket's decisions, then
  // come helper 1 of every bucket, helper 2, ...
  const int HLP = HELP ? a.pass_h : 0;  // launches without helpers compile none of their code
  const int role = HLP ? (int)(blockIdx.x / a.nbk) : 0;
  const int64_t bl = HLP ? (int64_t)(blockIdx.x % a.nbk) : (int64_t)blockIdx.x;
  const int64_t bucket = a.b0 + bl;
  const int64_t s = bucket / a.G;
  const int64_t t = bucket % a.G;
  const int N = a.N;
  const int P = N >> 1;
  const int NT = (N + 15) >> 4;
  const int nblk = (P + BP - 1) / BP;
  const int nch = (P + 63) >> 6;
  const int32_t* rows_in = a.idx_in ? a.idx_in + s * in_stride(a) + t * (int64_t)N : nullptr;
  const int64_t row_base = t * (int64_t)N;
  const float* Ub = a.U + s * a.u_slice + bucket_u(a, t, P);
  uint8_t* trace = a.trace ? a.trace + s * a.u_slice + bucket_u(a, t, P) : nullptr;
  int32_t* out = a.idx_out + s * out_stride(a) + t * (int64_t)P;
  const int64_t pb = s * (a.n_r >> 1) + t * (int64_t)P;
  const float* Eb = a.E + bl * a.e_tiles * (int64_t)TILE;
  // a valid address for the row loads of round 0 (their values are replaced)
  const int32_t* rsrc = rows_in ? rows_in : reinterpret_cast<const int32_t*>(Ub);

  extern __shared__ __align__(16) unsigned char smem[];
  double* s_alpha = reinterpret_cast<double*>(smem);
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(smem + L::mask_off(P));
  int* s_cnt = reinterpret_cast<int*>(smem + L::flag_off(P));  // decided, staged, rows[BW]
  auto slot = [&](int m) { return smem + L::slot_off(P) + (size_t)(m % L::NSLOT) * L::kSlot; };
  // slot fields
  auto sl_thr = [&](unsigned char* b) { return reinterpret_cast<double*>(b); };
  auto sl_rows = [&](unsigned char* b) { return reinterpret_cast<int32_t*>(b + BP * 8); };
  auto sl_own = [&](unsigned char* b) { return reinterpret_cast<u32x4*>(b + BP * 8 + 2 * BP * 4); };
  auto sl_next = [&](unsigned char* b) { return reinterpret_cast<u32x4*>(b + BP * 8 + 2 * BP * 4 + BP * L::CW * 16); };

  float* s_h2 = reinterpret_cast<float*>(smem + L::h2_off(P));
  float* s_mB = reinterpret_cast<float*>(smem + L::mb_off(P));
  for (int p = threadIdx.x; p < P; p += 64 * (BW + 2)) {
    s_alpha[p] = 0.0;
    s_h2[p] = a.h2[pb + p];
  }
  for (int b = threadIdx.x; b < nblk; b += 64 * (BW + 2)) s_mB[b] = a.mB[bucket * nblk + b];
  int* s_chunk = reinterpret_cast<int*>(smem + L::chunk_off(P));
  for (int c = threadIdx.x; c < (P + 63) / 64; c += 64 * (BW + 2)) s_chunk[c] = 0;
  if (threadIdx.x < 16) s_cnt[threadIdx.x] = threadIdx.x < 2 ? -1 : 0;
  __syncthreads();

  // Signed sum of a column's BP scores (decision bits in SMASK).
#define PASS_SUM(SRC, SMASK, SUM)                                                       \
  do {                                                                                 \
    SUM = 0.0f;                                                                        \
    _Pragma("unroll") for (int q_ = 0; q_ < QW; ++q_) {                                \
      const float e_[4] = {__uint_as_float(SRC[q_].x), __uint_as_float(SRC[q_].y),     \
                           __uint_as_float(SRC[q_].z), __uint_as_float(SRC[q_].w)};    \
      _Pragma("unroll") for (int c_ = 0; c_ < 4; ++c_)                                 \
        SUM += (((SMASK) >> (4 * q_ + c_)) & 1u) ? -e_[c_] : e_[c_];                   \
    }                                                                                  \
  } while (0)
  // Column of pair P_ in block B's score panel (P_ at or after block B).
#define PASS_COL(B, P_)                                                                 \
  reinterpret_cast<const u32x4*>(Eb + (panel_tiles(B, NT, RT) + ((P_) >> 3) - (B) * RT) * TILE + \
                                 ((P_) & 7) * BP)

  if (role > 0) {
    // ---- helper (waves 2..): the early rows of chunks ----
    // Helper wave hw of T = HLP BW takes chunks c = hw, hw + T, ... whose
    // hand_row(c) >= 0 and that it claims first (the bucket's workgroup
    // claims a chunk it reaches unclaimed and adds all its rows itself, so a
    // helper that is not resident delays nothing), rows 0 .. hand_row(c) in
    // order (a row's decisions from gmask, read with the row's scores and
    // checked by their tag), into a float64 alpha per pair in a register:
    // the same additions in the same order as the bucket's own bulk waves.
    // Then the chunk's partials go to galpha and, once written (vmcnt(0)),
    // its flag to "done".  All at agent scope: the bucket's workgroup runs on
    // another compute unit.
    if (wave < 2) return;
    const int T = HLP * BW;
    const int hw = (role - 1) * BW + (wave - 2);
    uint64_t* gm = a.gmask + bl * nblk;
    uint32_t* gf = a.gflag + bl * nch;
    const uint32_t claimed = 2u * (uint32_t)a.pass_tag, done = claimed + 1u;
    // next item to load: row fb of chunk fc
    int fc = hw, fb = 0;
    auto h_enter = [&]() {  // from fc on, the first chunk with rows that this wave claims
      while (fc < nch && (hand_row(fc) < 0 || shared_max(gf + fc, claimed) >= claimed)) fc += T;
      fb = 0;
    };
    h_enter();
    u32x4* colbuf = reinterpret_cast<u32x4*>(smem + L::colbuf_off(P) + (size_t)(wave - 2) * L::kColBuf);
    auto h_fetch = [&](u32x4* dst, uint64_t& word, int& ib, int& ic) {
      const bool live = fc < nch;
      ib = fb;
      ic = live ? fc : nch;
      if constexpr (L::COAL) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          dst[k] = (live ? PASS_COL(fb, min(64 * fc + 8 * k + lane / QW, P - 1))
                         : PASS_COL(0, lane / QW))[lane % QW];
      } else {
        const u32x4* c_ = live ? PASS_COL(fb, min(64 * fc + lane, P - 1)) : PASS_COL(0, 0);
#pragma unroll
        for (int k = 0; k < 8; ++k) dst[k] = c_[k];
      }
      // lane 0's read, broadcast only when the item is used: the wave does
      // not wait for it here
      word = 0;
      if (lane == 0)
        word = __hip_atomic_fetch_add(gm + (live ? fb : 0), (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (live && ++fb > hand_row(fc)) {
        fc += T;
        h_enter();
      }
    };
    u32x4 cb[NCB][8];
    uint64_t mw[NCB];
    int ib[NCB], ic[NCB];
#pragma unroll
    for (int r = 0; r < NCB; ++r) h_fetch(cb[r], mw[r], ib[r], ic[r]);
    bool more = ic[0] < nch;
    double acc = 0.0;
    while (more) {
#pragma unroll
      for (int r = 0; r < NCB; ++r) {
        const int b = ib[r], c = ic[r];
        const bool live = c < nch;
        const uint64_t w0 = __shfl(mw[r], 0);
        const uint32_t smask = live ? decided_mask(gm + b, w0, helper_tag(a.pass_tag, b), a.status) : 0u;
        u32x4 col[QW];
        if constexpr (L::COAL) {
#pragma unroll
          for (int k = 0; k < 8; ++k) colbuf[(8 * k + lane / QW) * L::CW + lane % QW] = cb[r][k];
#pragma unroll
          for (int q = 0; q < QW; ++q) col[q] = colbuf[lane * L::CW + q];
        } else {
#pragma unroll
          for (int q = 0; q < QW; ++q) col[q] = cb[r][q];
        }
        float sum;
        PASS_SUM(col, smask, sum);
        const int p = 64 * c + lane;
        if (live && b == 0) acc = 0.0;
        if (live && p < P) acc += ldexp((double)sum, (int)scale_shift(s_mB[b], s_h2[p]));
        h_fetch(cb[r], mw[r], ib[r], ic[r]);
        if (live && b == hand_row(c)) {
          if (p < P) shared_write(a.galpha + bl * P + p, __double_as_longlong(acc));
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
          __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the partials are written
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
          (void)shared_max(gf + c, done);
        }
        more = ic[(r + 1) % NCB] < nch;
      }
    }
  } else if (wave == 0) {
    // ---- decider ----
    __builtin_amdgcn_s_setprio(3);  // ahead of the bulk waves sharing its SIMD
    double anear = 0.0;             // this lane's pair: the previous block's contribution
    for (int m = 0; m < nblk; ++m) {
      const int npb = min(BP, P - m * BP);
      wait_at_least(&s_cnt[1], m, a.status);
      // the bulk sums of blocks 0 .. m-2 are in this block's pairs (64-pair
      // chunk m / 2)
      if (m >= 2) wait_at_least(&s_chunk[m >> 1], m - 1, a.status);
      unsigned char* sb = slot(m);
      const int p = lane;
      const int pl = lane & (BP - 1);
      const bool active = p < npb;
      const int gp = m * BP + p;
      const double alpha_in = s_alpha[min(gp, P - 1)] + anear;
      // the block's own scores are at its shifted scale: decide there
      const float mBm = s_mB[m];
      const int sh = (int)scale_shift(mBm, s_h2[min(gp, P - 1)]);
      const double thr = ldexp(sl_thr(sb)[pl], -sh);
      const int32_t r0 = sl_rows(sb)[pl], r1 = sl_rows(sb)[BP + pl];
      double alpha = ldexp(alpha_in, -sh);
      // this pair's scores against the block's pairs, held in registers
      // before the loop (the loop is the decider's critical path and must
      // not wait on LDS); widened to float64 inside the loop, off the chain.
      // No masking: lane p's alpha is read only at its own decision (step
      // p), before any score of a pair i >= p has been added to it, and the
      // decisions of lanes past the block's last pair are dropped below.
      // The same for this block's scores against the next block's pair pl:
      // their signed sum (the next block's contribution from this block) is
      // accumulated inside the loop, in the order of the bulk sums.
      float ef[BP], en[BP];
      const u32x4* oc = sl_own(sb) + pl * L::CW;
      const u32x4* nc = sl_next(sb) + pl * L::CW;
      u32x4 xs[QW], xn[QW];
#pragma unroll
      for (int q = 0; q < QW; ++q) {
        xs[q] = oc[q];
        xn[q] = nc[q];
      }
#pragma unroll
      for (int q = 0; q < QW; ++q)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          ef[4 * q + c] = __uint_as_float(xs[q][c]);
          en[4 * q + c] = __uint_as_float(xn[q][c]);
          asm volatile("" : "+v"(ef[4 * q + c]), "+v"(en[4 * q + c]));
        }
      __builtin_amdgcn_sched_barrier(0);
      float near = 0.0f;
      const uint32_t smask = decide_block<true>(alpha, thr, ef, en, npb, near);
      if (lane == 0) s_mask[m] = smask;
      publish(&s_cnt[0], m);
      if (HLP && lane == 0)
        shared_write(a.gmask + bl * nblk + m, ((uint64_t)helper_tag(a.pass_tag, m) << 32) | smask);
      const uint32_t bit = (smask >> (p & 31)) & 1u;
      if (active) {
        out[gp] = bit ? r1 : r0;
        if (trace) trace[gp] = (uint8_t)bit;
      }
      // the next block's pairs take this block's signed scores
      anear = ldexp((double)near, (int)scale_shift(mBm, s_h2[min((m + 1) * BP + pl, P - 1)]));
    }
  } else if (wave == 1) {
    // ---- fetcher: block m's inputs into slot m % 3 ----
    // Lane l fetches word l%QW of the columns of pairs l/QW + 8r (r < 4) of
    // the block's own scores and of its scores against the next block; lanes
    // < BP also the pair terms, uniform and rows of pair l.  Lanes past a
    // block's last pair read that pair's inputs.  One block is fetched while
    // the previous one is staged.
    __builtin_amdgcn_s_setprio(2);
    u32x4 fo[FD][4], fn[FD][4];
    float flbt[FD], fh2[FD], fu[FD];
    int32_t fr0[FD], fr1[FD];
#define PASS_FETCH(B, K)                                                                \
  do {                                                                                 \
    const int b_ = min(B, nblk - 1);                                                   \
    const int npb_ = min(BP, P - b_ * BP);                                             \
    const float* e_ = Eb + panel_tiles(b_, NT, RT) * TILE;                             \
    _Pragma("unroll") for (int r_ = 0; r_ < 4; ++r_) {                                 \
      const int pc_ = min(lane / QW + 8 * r_, npb_ - 1);                               \
      fo[K][r_] = reinterpret_cast<const u32x4*>(e_ + (pc_ >> 3) * TILE + (pc_ & 7) * BP)[lane % QW]; \
      /* next block's pairs (the last block reads its own last column) */           \
      const int pn_ = min((b_ + 1) * BP + lane / QW + 8 * r_, P - 1);                  \
      fn[K][r_] = PASS_COL(b_, pn_)[lane % QW];                                        \
    }                                                                                  \
    const int gp_ = b_ * BP + min(lane & (BP - 1), npb_ - 1);                          \
    flbt[K] = a.lbt[pb + gp_];                                                         \
    fh2[K] = a.h2[pb + gp_];                                                           \
    fu[K] = Ub[gp_];                                                                   \
    fr0[K] = rsrc[rows_in ? 2 * gp_ : 0];                                              \
    fr1[K] = rsrc[rows_in ? 2 * gp_ + 1 : 0];                                          \
  } while (0)
    double carry = -INFINITY;  // log b_max over the pairs of earlier blocks
#define PASS_STAGE(B, K)                                                                \
  do {                                                                                 \
    const int npb_ = min(BP, P - (B) * BP);                                            \
    const double thr_ = block_threshold(flbt[K], fh2[K], fu[K], npb_, lane, a.log_c, carry); \
    /* slot B % NSLOT held block B - NSLOT, left once B - NSLOT + 1 is decided */    \
    if ((B) >= L::NSLOT) wait_at_least(&s_cnt[0], (B) - (L::NSLOT - 1), a.status);    \
    unsigned char* sb_ = slot(B);                                                      \
    _Pragma("unroll") for (int r_ = 0; r_ < 4; ++r_) {                                 \
      sl_own(sb_)[(lane / QW + 8 * r_) * L::CW + lane % QW] = fo[K][r_];               \
      sl_next(sb_)[(lane / QW + 8 * r_) * L::CW + lane % QW] = fn[K][r_];              \
    }                                                                                  \
    if (lane < BP) {                                                                   \
      sl_thr(sb_)[lane] = thr_;                                                        \
      sl_rows(sb_)[lane] = rows_in ? fr0[K] : (int32_t)(row_base + 2 * ((B) * BP + lane)); \
      sl_rows(sb_)[BP + lane] = rows_in ? fr1[K] : (int32_t)(row_base + 2 * ((B) * BP + lane) + 1); \
    }                                                                                  \
    publish(&s_cnt[1], B);                                                             \
  } while (0)
    // FD blocks' loads in flight: block m is staged from register set m % FD,
    // which then takes the loads of block m + FD
#pragma unroll
    for (int k = 0; k < FD; ++k) PASS_FETCH(k, k);
    for (int m = 0; m < nblk; m += FD) {
#pragma unroll
      for (int k = 0; k < FD; ++k) {
        if (m + k < nblk) PASS_STAGE(m + k, k);
        PASS_FETCH(m + k + FD, k);
      }
    }
#undef PASS_FETCH
#undef PASS_STAGE
  } else {
    // ---- bulk updates, blocks 0 .. nblk-3 ----
    // Bulk wave w = wave-2 owns the 64-pair chunks c = w, w + BW, ... of the
    // bucket (blocks 2c, 2c+1).  Row b (block b's signed scores) adds to the
    // pairs of block b+2 on, so chunk c takes rows 0 .. 2c-1 (row 2c-1 only
    // in its second block).  A wave's items are (row, chunk) chunk by chunk
    // in increasing c, rows in order within a chunk: items are taken in the
    // order the decider needs them (chunk c before block 2c), and a chunk's
    // progress does not wait for the wave's later chunks.  The items form one
    // stream held in an NCB-slot register ring (with each slot's row and
    // chunk): each consumed slot is refilled at once with the item NCB later,
    // so the loads run ahead whatever the decisions.  Lane l sums column l of
    // the chunk in ascending order (the order of the decider's sums); with
    // COAL the chunk is loaded a score tile (8 columns, 1 KiB) per
    // instruction, 8 lanes to a column, and turned through the wave's LDS
    // column buffer.  After row b of chunk c the wave publishes b + 1 in
    // s_chunk[c] (rows completed).  With helpers, a chunk a helper has
    // claimed starts from the helper's partial alpha over rows
    // 0 .. hand_row(c) (taken from galpha once the chunk's flag is "done")
    // and continues with rows hand_row(c) + 1 on; a chunk the wave reaches
    // unclaimed it claims and takes whole.
    const int w = wave - 2;
    const int nrow = nblk - 2;
    auto last_row = [&](int c) { return min(2 * c - 1, nrow - 1); };  // < 0: no item
    uint32_t* gf = HLP ? a.gflag + bl * nch : nullptr;
    const uint32_t claimed = 2u * (uint32_t)a.pass_tag, done = claimed + 1u;
    // next item to load: row fb of chunk fc; fh: fb is the first row after
    // a helper's partial
    int fc = w, fb = 0;
    bool fh = false;
    auto enter = [&]() {  // from fc on, the first chunk with items
      while (fc < nch && last_row(fc) < 0) fc += BW;
      fb = 0;
      fh = false;
      if (fc < nch && HLP && hand_row(fc) >= 0 && shared_max(gf + fc, claimed) >= claimed) {
        fb = hand_row(fc) + 1;
        fh = true;
      }
    };
    enter();
    u32x4* colbuf = reinterpret_cast<u32x4*>(smem + L::colbuf_off(P) + (size_t)w * L::kColBuf);
    auto fetch_next = [&](u32x4* dst, int& ib, int& ic, bool& ih) {
      const bool live = fc < nch;
      ib = fb;
      ic = live ? fc : nch;
      ih = live && fh;
      fh = false;
      // COAL: word lane % QW of column 8 k + lane / QW of the chunk; else
      // word k of column lane (past the stream's end: valid columns, never
      // used)
      if constexpr (L::COAL) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          dst[k] = (live ? PASS_COL(fb, min(64 * fc + 8 * k + lane / QW, P - 1))
                         : PASS_COL(0, lane / QW))[lane % QW];
      } else {
        const u32x4* c_ = live ? PASS_COL(fb, min(64 * fc + lane, P - 1)) : PASS_COL(0, 0);
#pragma unroll
        for (int k = 0; k < 8; ++k) dst[k] = c_[k];
      }
      if (live && ++fb > last_row(fc)) {
        fc += BW;
        enter();
      }
    };
    u32x4 cb[NCB][8];
    int ib[NCB], ic[NCB];
    bool ih[NCB];
#pragma unroll
    for (int r = 0; r < NCB; ++r) fetch_next(cb[r], ib[r], ic[r], ih[r]);
    int decided = -1;  // last decided block seen
    bool more = ic[0] < nch;
    // Every slot of a turn is used and refilled whether or not the stream
    // has ended (loads past the end are of valid columns, nothing is added):
    // all paths then issue the same loads, and the wait before a slot's use
    // is for that slot's loads only.
    while (more) {
#pragma unroll
      for (int r = 0; r < NCB; ++r) {
        const int b = ib[r], c = ic[r];
        const bool live = c < nch;
        if (live && ih[r]) {
          // the helper's partial alpha of the chunk's pairs (rows 0 .. hand_row(c))
          wait_flag(gf + c, done, a.status);
          __atomic_signal_fence(__ATOMIC_SEQ_CST);
          const int pc = 64 * c + lane;
          if (pc < P)
            s_alpha[pc] = __longlong_as_double((long long)shared_read_lane(a.galpha + bl * P + pc));
          publish(&s_chunk[c], hand_row(c) + 1);
        }
        if (live && decided < b) decided = wait_at_least(&s_cnt[0], b, a.status);
        const uint32_t smask = s_mask[live ? b : 0];
        u32x4 col[QW];
        if constexpr (L::COAL) {
#pragma unroll
          for (int k = 0; k < 8; ++k) colbuf[(8 * k + lane / QW) * L::CW + lane % QW] = cb[r][k];
#pragma unroll
          for (int q = 0; q < QW; ++q) col[q] = colbuf[lane * L::CW + q];
        } else {
#pragma unroll
          for (int q = 0; q < QW; ++q) col[q] = cb[r][q];
        }
        float sum;
        PASS_SUM(col, smask, sum);
        const int p = 64 * c + lane;
        if (live && p >= (b + 2) * BP && p < P)
          s_alpha[p] += ldexp((double)sum, (int)scale_shift(s_mB[b], s_h2[p]));
        fetch_next(cb[r], ib[r], ic[r], ih[r]);
        if (live) publish(&s_chunk[c], b + 1);
        more = ic[(r + 1) % NCB] < nch;
      }
    }
  }
#undef PASS_SUM
#undef PASS_COL
}

// Gram of rows [0,16) against rows [16,32) through the fragment path used by
// the score kernel (lane-layout self-check).
template <typename T, int D>
__global__ __launch_bounds__(64) void gram16_kernel(const T* rows, float* out) {
  constexpr int NV = Frag<T, D>::NV;
  const int lane = threadIdx.x, m16 = lane & 15, g = lane >> 4;
  uint4 a[NV], b[NV];
  load_frag<T, D>(rows, m16, g, true, a);
  load_frag<T, D>(rows, 16 + m16, g, true, b);
  floatx4_t acc = {0.f, 0.f, 0.f, 0.f};
  acc = mma_rows<T, D>(a, b, acc);
#pragma unroll
  for (int i = 0; i < 4; ++i) out[(4 * g + i) * 16 + m16] = acc[i];
}

// Buckets interleaved per XCD in a score launch (at most the XCD's share):
// enough to stagger the workgroups' ends, few enough that their rows stay in
// the XCD's L2.
#ifndef SCORE_IL
#define SCORE_IL 16
#endif
template <typename T, int D>
hipError_t launch_scores_td(const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  constexpr int WO = score_waves<T, D>();
  using SS = ScoreShape<T, D, WO>;  // own and streamed chunks share the groups
  auto kern_mixed = pair_scores_kernel<T, D, false, false, WO>;
  auto kern_own = pair_scores_kernel<T, D, false, true, WO>;
  const size_t lds = SS::LDS, lds_own = SS::LDS;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern_mixed),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (lds_own > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern_own),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_own);
    if (e != hipSuccess) return e;
  }
  const int64_t NT = (a0.N + 15) / 16;
  const int64_t groups = (NT + SS::GT - 1) / SS::GT;
  const int64_t rest = NT > SS::GT ? NT - SS::GT : 0;  // tiles after the first group
  // Column tiles per streamed chunk (one workgroup's tiles, taken one after
  // the other): kScoreChunkLong while the launch keeps at least four
  // workgroups per CU (each workgroup loads its group's fragments once, for
  // more tiles), else kScoreChunk, or fewer when the launch would leave the
  // device short of workgroups (a few large buckets: each chunk's tiles are
  // then the launch's critical path)
  HalveArgs a = a0;
  auto workgroups = [&](int64_t c) {
    int64_t w = 0;
    for (int64_t g = 0; g < groups; ++g) {
      const int64_t rest_g = NT - (g + 1) * SS::GT;
      w += 1 + (rest_g > 0 ? (rest_g + c - 1) / c : 0);
    }
    return w * nbk;
  };
  if (workgroups(kScoreChunkLong) >= kScoreLongWorkgroups) a.ch = kScoreChunkLong;
  for (const int c : {15, 9, 6})
    if (workgroups(a.ch) <= kScoreMinWorkgroups && c < a.ch) a.ch = c;
  const int64_t nch = 1 + (rest + a.ch - 1) / a.ch;
  // one workgroup per (bucket, group, chunk) with work, buckets padded to a
  // multiple of the eight XCDs (the padding workgroups return at once)
  auto launch = [&](HalveArgs x, int chunk0, int nz) {
    x.chunk0 = chunk0;
    x.nz = nz;
    x.ngrp = (int32_t)groups;
    x.nbk = nbk;
    int64_t ipb = 0;
    for (int64_t g = 0; g < groups; ++g) {
      const int64_t rest_g = NT - (g + 1) * SS::GT;
      const int64_t nsc = rest_g > 0 ? (rest_g + a.ch - 1) / a.ch : 0;
      ipb += std::max<int64_t>(0, std::min<int64_t>(chunk0 + nz, 1 + nsc) - chunk0);
    }
    x.ipb = (int32_t)ipb;
    x.il = (int32_t)std::min<int64_t>(SCORE_IL, (nbk + 7) / 8);
    const int64_t per_xcd = ((nbk + 7) / 8 + x.il - 1) / x.il * x.il;
    const int64_t wgs = 8 * per_xcd * ipb;
    // a launch of own chunks only takes the own-only instantiation
    if (chunk0 == 0 && nz == 1)
      hipLaunchKernelGGL(kern_own, dim3((unsigned)wgs), dim3(64 * WO), lds_own, st, x);
    else
      hipLaunchKernelGGL(kern_mixed, dim3((unsigned)wgs), dim3(64 * WO), lds, st, x);
  };
  if (a.rowh2_write && nch > 1) {
    // the streamed chunks read the row scales the own chunks write: two launches
    launch(a, 0, 1);
    HalveArgs rest_a = a;
    rest_a.rowh2_write = 0;
    launch(rest_a, 1, (int)(nch - 1));
    return hipGetLastError();
  }
  launch(a, 0, (int)nch);
  return hipGetLastError();
}

// One wave per bucket for buckets of up to 16 RT rows whose fragments fit
// (RT NV <= 16 words per lane and operand).
template <typename T, int D>
constexpr int tiny_tiles() {
  return Frag<T, D>::NV <= 4 ? 4 : 16 / Frag<T, D>::NV;
}

template <typename T, int D, int RT>
hipError_t launch_tiny_td(const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  HalveArgs a = a0;
  a.nbk = nbk;
  const unsigned wgs = (unsigned)((nbk + kTinyWaves - 1) / kTinyWaves);
  hipLaunchKernelGGL((tiny_halve_kernel<T, D, RT>), dim3(wgs), dim3(64 * kTinyWaves), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_local_td(const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  // with few buckets one wave per bucket leaves the GPU idle and a bucket's
  // latency (its tiles one after another) sets the time: the local kernel's
  // eight waves per bucket are faster there
  if (nbk >= kTinyMinBuckets) {
    if (a0.N <= 16) return launch_tiny_td<T, D, 1>(a0, nbk, st);
    if constexpr (tiny_tiles<T, D>() >= 2)
      if (a0.N <= 32) return launch_tiny_td<T, D, 2>(a0, nbk, st);
    if constexpr (tiny_tiles<T, D>() >= 4)
      if (a0.N <= 64) return launch_tiny_td<T, D, 4>(a0, nbk, st);
  }
  constexpr int WO = score_waves<T, D>();
  using SS = ScoreShape<T, D, WO>;
  auto kern = pair_scores_kernel<T, D, true, true, WO>;
  const int64_t NT = (a0.N + 15) / 16, nb = (a0.N + 63) / 64, P = a0.N / 2;
  // stages, score tiles, pair scale exponents of the rows, staged row
  // scales, half-block row scale maxima, pair terms [2][P], then (8-byte
  // aligned) the decisions' thresholds and alphas [2][BLOCKS][64] and masks
  const size_t lds = (size_t)kScoreStages * SS::CHUNKS * 1024 +
                     (size_t)panel_tiles(nb, NT, 4) * kETileLds * 4 + SS::GT * 16 * 4 +
                     kScoreStages * 16 * 4 + 2 * SS::BLOCKS * 4 + 2 * P * 4 + 8 +
                     2 * 64 * SS::BLOCKS * 8 + SS::BLOCKS * 4;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  HalveArgs a = a0;
  a.chunk0 = 0;
  a.ch = kScoreChunk;
  a.e_tiles = 0;
  hipLaunchKernelGGL(kern, dim3((unsigned)nbk), dim3(64 * WO), lds, st, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_local_t(int64_t d, const HalveArgs& a, int64_t nbk, hipStream_t st) {
  switch (d) {
    case 32: return launch_local_td<T, 32>(a, nbk, st);
    case 64: return launch_local_td<T, 64>(a, nbk, st);
    case 128: return launch_local_td<T, 128>(a, nbk, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
int64_t local_rows_t(int64_t d) {
  switch (d) {
    case 32: return ScoreShape<T, 32, score_waves<T, 32>()>::GT * 16;
    case 64: return ScoreShape<T, 64, score_waves<T, 64>()>::GT * 16;
    case 128: return ScoreShape<T, 128, score_waves<T, 128>()>::GT * 16;
    default: return 0;
  }
}

template <typename T>
hipError_t launch_scores_t(int64_t d, const HalveArgs& a, int64_t nbk, hipStream_t st) {
  switch (d) {
    case 32: return launch_scores_td<T, 32>(a, nbk, st);
    case 64: return launch_scores_td<T, 64>(a, nbk, st);
    case 128: return launch_scores_td<T, 128>(a, nbk, st);
    default: return hipErrorInvalidValue;
  }
}

// Helper workgroups per bucket for a decision launch: rounds of at most
// kHelperMaxBuckets buckets of at least kHelperMinPairs pairs (one launch
// per round: the tags of gmask and gflag are per round), as many as the
// device's compute units hold beside the buckets' own, at most kMaxHelpers.
int pass_helpers(const HalveArgs& a, int64_t nbk) {
  const int64_t P = a.N / 2;
  if (!a.gmask || !a.gflag || !a.galpha || a.pass_tag <= 0 || a.b0 != 0) return 0;
  // helper k of bucket b is workgroup k nbk + b: on the bucket's XCD (the
  // dispatcher deals workgroups to the 8 XCDs in turn) when 8 divides nbk
  if (P < kHelperMinPairs || P % 64 != 0 || nbk < 1 || nbk > kHelperMaxBuckets || nbk % 8 != 0) return 0;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const int64_t h = cus / nbk - 1;
  return (int)(h < 0 ? 0 : (h > kMaxHelpers ? kMaxHelpers : h));
}

template <int BW, int NCB, int FD, bool HELP>
hipError_t launch_pass_k(const HalveArgs& a, int64_t grid, hipStream_t st) {
  const size_t lds = PassLds<BW, NCB, FD>::bytes((int)(a.N / 2));
  auto kern = halve_pass_kernel<BW, NCB, FD, HELP>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * (BW + 2)), lds, st, a);
  return hipGetLastError();
}

// HELPERS: the shape may take decision helpers (the large shapes).  Helpers
// follow the buckets' own workgroups in the grid; a helper waits only for
// decisions, and a bucket's workgroup never waits for a helper that has not
// claimed a chunk, so any residency order completes.
template <int BW, int NCB, int FD, bool HELPERS = false>
hipError_t launch_pass_w(const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  HalveArgs a = a0;
  a.nbk = nbk;
  a.pass_h = 0;
  if constexpr (HELPERS) {
    a.pass_h = pass_helpers(a, nbk);
    if (a.pass_h > 0) return launch_pass_k<BW, NCB, FD, true>(a, nbk * (1 + a.pass_h), st);
  }
  return launch_pass_k<BW, NCB, FD, false>(a, nbk, st);
}

}  // namespace

int64_t halve_score_tiles(int64_t N) {
  const int64_t NT = (N + 15) / 16;
  const int64_t nb = (N + 63) / 64;
  return panel_tiles(nb, NT, 4);
}

size_t halve_score_bytes(int64_t N) {
  return (size_t)halve_score_tiles(N) * 8 * 32 * 4;  // tiles of 8 columns x 32 rows, float32
}

static HalveArgs with_layout(const HalveArgs& a0) {
  HalveArgs a = a0;
  a.ch = kScoreChunk;
  a.e_tiles = halve_score_tiles(a.N);
  return a;
}

hipError_t launch_scores(int dtype, int64_t d, const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  const HalveArgs a = with_layout(a0);
  return dtype == 0 ? launch_scores_t<float>(d, a, nbk, st) : launch_scores_t<bf16_t>(d, a, nbk, st);
}

int64_t halve_local_rows(int dtype, int64_t d) {
  return dtype == 0 ? local_rows_t<float>(d) : local_rows_t<bf16_t>(d);
}

hipError_t launch_local(int dtype, int64_t d, const HalveArgs& a, int64_t nbk, hipStream_t st) {
  if (a.N > halve_local_rows(dtype, d)) return hipErrorInvalidValue;
  return dtype == 0 ? launch_local_t<float>(d, a, nbk, st) : launch_local_t<bf16_t>(d, a, nbk, st);
}

// Decision pass shapes <bulk waves, chunks in flight per bulk wave, blocks in
// flight in the fetcher> for small (<= 256 pairs after the first two
// blocks), medium (<= 512) and large buckets.  Large buckets run one per CU
// (64 buckets of 2048 rows on the long workload), where ten bulk waves keep
// the decider fed (round 3 there: 69.7 -> 58.7 us against six); a deeper
// fetcher gained nothing.
#ifndef PASS_FD_S
#define PASS_FD_S 2
#endif
#ifndef PASS_BW_M
#define PASS_BW_M 6
#define PASS_NCB_M 3
#define PASS_FD_M 2
#endif
#ifndef PASS_BW_L
#define PASS_BW_L 10
#define PASS_NCB_L 3
#define PASS_FD_L 2
#endif
constexpr size_t kPassMaxLds = (size_t)160 << 10;  // LDS of a gfx950 CU
hipError_t launch_decide(const HalveArgs& a0, int64_t nbk, hipStream_t st) {
  const HalveArgs a = with_layout(a0);
  // bulk waves x prefetched chunks x 64 pairs should cover the pairs after
  // the first two blocks
  const int64_t later = a.N / 2 - 64;
  if (later <= 64) return launch_pass_w<1, 1, PASS_FD_S>(a, nbk, st);
  if (later <= 256) return launch_pass_w<2, 2, PASS_FD_S>(a, nbk, st);
  if (later <= 512) return launch_pass_w<PASS_BW_M, PASS_NCB_M, PASS_FD_M>(a, nbk, st);
  // the large shape's column buffers take 9 KiB of LDS per bulk wave: past
  // the 160 KiB of a CU (buckets above 4096 rows) eight bulk waves run, past
  // that the medium shape
  if (PassLds<PASS_BW_L, PASS_NCB_L, PASS_FD_L>::bytes((int)(a.N / 2)) <= kPassMaxLds)
    return launch_pass_w<PASS_BW_L, PASS_NCB_L, PASS_FD_L, true>(a, nbk, st);
  if (PassLds<8, 3, 2>::bytes((int)(a.N / 2)) <= kPassMaxLds)
    return launch_pass_w<8, 3, 2, true>(a, nbk, st);
  return launch_pass_w<PASS_BW_M, PASS_NCB_M, PASS_FD_M, true>(a, nbk, st);
}

hipError_t launch_vmax(int dtype, const void* V, int64_t S, int64_t n, int64_t ld, int64_t d,
                       uint32_t* vmax_bits, hipStream_t st, int32_t* status, int64_t zero_words) {
  const int64_t zw = zero_words > S ? zero_words : S;
  hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)((zw + 255) / 256)), dim3(256), 0, st,
                     vmax_bits, zw, status);
  const int64_t bytes = dtype == 0 ? 4 : 2;
  const int64_t words = n * d * bytes / 16, slice_words = ld * d * bytes / 16;
  // 256 KiB of V per workgroup, less for small inputs so that the scan has
  // about 1024 workgroups (one workgroup reads ~40 GB/s; 64 of them made the
  // ViT-like workload's scan take 13 us), in whole turns of the 8-load loop
  constexpr int64_t kVmaxTurn = 8 * 256;
  int64_t per_block = 16384;
  const int64_t want = (words * S + 1023) / 1024;
  if (want < per_block) per_block = std::max<int64_t>(kVmaxTurn, (want + kVmaxTurn - 1) / kVmaxTurn * kVmaxTurn);
  const int64_t chunks = (words + per_block - 1) / per_block;
  dim3 grid((unsigned)chunks, (unsigned)S);
  if (dtype == 0)
    hipLaunchKernelGGL(vmax_kernel<float>, grid, dim3(256), 0, st, (const float*)V, words,
                       slice_words, per_block, vmax_bits);
  else
    hipLaunchKernelGGL(vmax_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)V, words,
                       slice_words, per_block, vmax_bits);
  return hipGetLastError();
}

hipError_t launch_subsample(int64_t S, int64_t n, int64_t n_kept, const float* U,
                            int64_t u_slice, int32_t* idx0, hipStream_t st) {
  dim3 grid((unsigned)((n_kept + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(subsample_kernel, grid, dim3(256), 0, st, n, n_kept, U, u_slice, idx0);
  return hipGetLastError();
}

hipError_t launch_fill_rows(int64_t S, int64_t n_out, const int32_t* src, int64_t src_stride,
                            int32_t* dst, hipStream_t st) {
  dim3 grid((unsigned)((n_out + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(fill_rows_kernel, grid, dim3(256), 0, st, n_out, src, src_stride, dst);
  return hipGetLastError();
}

hipError_t launch_assemble(int64_t S, int64_t n, int64_t ns, int64_t n_out, int64_t nw,
                           const int32_t* src, int64_t src_stride, int32_t* dst, float* logw,
                           float lw_core, hipStream_t st) {
  const int64_t m = ns + n_out + nw;
  dim3 grid((unsigned)((m + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(assemble_kernel, grid, dim3(256), 0, st, n, ns, n_out, nw, src, src_stride,
                     dst, logw, lw_core);
  return hipGetLastError();
}

// Uniform halving: pair p of slice s keeps idx_in[2p+1] iff u < 1/2, else
// idx_in[2p] (idx_in null = the identity).  The pairs of a round are
// consecutive in the slice's current order, bucket after bucket, as are
// their draws, so the buckets need no separate treatment.
// With u_bucket, bucket t (N rows, N/2 pairs) draws from u_bucket[t] on; the
// lists are in_stride / out_stride apart per slice (0: packed).
__global__ void uniform_halve_kernel(int64_t n_r, const int32_t* idx_in, const float* U,
                                     int64_t u_slice, int64_t u_off, int32_t* idx_out,
                                     uint8_t* trace, int64_t N, const int64_t* u_bucket,
                                     int64_t in_stride, int64_t out_stride) {
  const int64_t s = blockIdx.y;
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t P = n_r >> 1;
  if (p >= P) return;
  const int64_t ui =
      s * u_slice + (u_bucket ? u_bucket[p / (N >> 1)] + p % (N >> 1) : u_off + p);
  const int swap = U[ui] < 0.5f;
  const int64_t j = 2 * p + swap;
  idx_out[s * (out_stride ? out_stride : P) + p] =
      idx_in ? idx_in[s * (in_stride ? in_stride : n_r) + j] : (int32_t)j;
  if (trace) trace[ui] = (uint8_t)swap;
}

hipError_t launch_uniform_halve(int64_t S, int64_t n_r, const int32_t* idx_in, const float* U,
                                int64_t u_slice, int64_t u_off, int32_t* idx_out,
                                uint8_t* trace, hipStream_t st, int64_t N,
                                const int64_t* u_bucket, int64_t in_stride, int64_t out_stride) {
  const int64_t P = n_r / 2;
  dim3 grid((unsigned)((P + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(uniform_halve_kernel, grid, dim3(256), 0, st, n_r, idx_in, U, u_slice,
                     u_off, idx_out, trace, N > 0 ? N : n_r, u_bucket, in_stride, out_stride);
  return hipGetLastError();
}

// Every round of uniform halving of one slice per workgroup, the slice's
// indices held in LDS (n_kept <= kUniformFusedRows): in round r each thread
// reads its pairs' kept indices, the workgroup synchronises, and the halved
// list is written back in place.
constexpr int kUniformThreads = 1024;
constexpr int64_t kUniformFusedRows = 32768;
__global__ __launch_bounds__(kUniformThreads) void uniform_compress_kernel(
    int64_t n_kept, int32_t L, const int32_t* idx0, const float* U, int64_t u_slice,
    int64_t u_off0, int32_t* idx_out, int64_t n_out, uint8_t* trace) {
  extern __shared__ int32_t s_idx[];
  constexpr int PPT = (int)(kUniformFusedRows / 2 / kUniformThreads);  // pairs per thread, round 0
  const int64_t s = blockIdx.x;
  const int tid = threadIdx.x;
  for (int64_t i = tid; i < n_kept; i += kUniformThreads)
    s_idx[i] = idx0 ? idx0[s * n_kept + i] : (int32_t)i;
  __syncthreads();
  int64_t n_r = n_kept, u_off = u_off0;
  for (int32_t r = 0; r < L; ++r) {
    const int64_t P = n_r >> 1;
    int32_t keep[PPT];
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int64_t p = tid + (int64_t)k * kUniformThreads;
      if (p < P) {
        const int64_t ui = s * u_slice + u_off + p;
        const int swap = U[ui] < 0.5f;
        keep[k] = s_idx[2 * p + swap];
        if (trace) trace[ui] = (uint8_t)swap;
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int64_t p = tid + (int64_t)k * kUniformThreads;
      if (p < P) s_idx[p] = keep[k];
    }
    __syncthreads();
    n_r = P;
    u_off += P;
  }
  for (int64_t i = tid; i < n_out; i += kUniformThreads) idx_out[s * n_out + i] = s_idx[i];
}

bool uniform_fused_ok(int64_t n_kept) { return n_kept <= kUniformFusedRows; }

hipError_t launch_uniform_compress(int64_t S, int64_t n_kept, int32_t L, const int32_t* idx0,
                                   const float* U, int64_t u_slice, int64_t u_off0,
                                   int32_t* idx_out, int64_t n_out, uint8_t* trace,
                                   hipStream_t st) {
  if (!uniform_fused_ok(n_kept)) return hipErrorInvalidValue;
  const size_t lds = (size_t)n_kept * 4;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(uniform_compress_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(uniform_compress_kernel, dim3((unsigned)S), dim3(kUniformThreads), lds, st,
                     n_kept, L, idx0, U, u_slice, u_off0, idx_out, n_out, trace);
  return hipGetLastError();
}

hipError_t launch_zero_status(int32_t* status, hipStream_t st) {
  hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(64), 0, st, nullptr, 0, status);
  return hipGetLastError();
}

hipError_t launch_zero_u8(uint8_t* p, int64_t count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u8_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, p,
                     count);
  return hipGetLastError();
}

hipError_t launch_gram16(int dtype, int64_t d, const void* rows, float* out, hipStream_t st) {
  dim3 grid(1), block(64);
#define THIN_G16(T, DD) \
  hipLaunchKernelGGL((gram16_kernel<T, DD>), grid, block, 0, st, (const T*)rows, out)
  if (dtype == 0) {
    if (d == 32) THIN_G16(float, 32);
    else if (d == 64) THIN_G16(float, 64);
    else if (d == 128) THIN_G16(float, 128);
    else return hipErrorInvalidValue;
  } else {
    if (d == 32) THIN_G16(bf16_t, 32);
    else if (d == 64) THIN_G16(bf16_t, 64);
    else if (d == 128) THIN_G16(bf16_t, 128);
    else return hipErrorInvalidValue;
  }
#undef THIN_G16
  return hipGetLastError();
}

}  // namespace thin
