// Compress path on gfx950: v_max scan, stratified subsample and the bucketed
// kernel-halving round (KH(1/2) under kappa_att), one launch per round.
#include <math.h>

#include "common.hpp"
#include "launch.hpp"

namespace thin {

namespace {

constexpr double kLn2 = 0.69314718055994530942;
constexpr double kLog2e = 1.44269504088896340736;
// Cross-term exponents (base 2) are clamped here; they exceed the column
// pair's own diagonal exponent only for data far outside attention ranges.
constexpr float kExpClamp = 64.0f;

__device__ __forceinline__ float wave_max_f(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// ---------------------------------------------------------------------------
// v_max = max_i ||v_i||_inf over all n rows of a slice (Sec. 2.1, eq. katt).
// grid (chunks, S); the per-slice maximum is merged with an integer atomicMax
// on the float's bit pattern (valid for non-negative floats).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void vmax_kernel(const T* V, int64_t words_per_slice,
                                                   int64_t words_per_block, uint32_t* vmax_bits) {
  const int64_t s = blockIdx.y;
  const uint4* base = reinterpret_cast<const uint4*>(V) + s * words_per_slice;
  int64_t w0 = (int64_t)blockIdx.x * words_per_block;
  int64_t w1 = w0 + words_per_block;
  if (w1 > words_per_slice) w1 = words_per_slice;
  float m = 0.0f;
  for (int64_t w = w0 + threadIdx.x; w < w1; w += blockDim.x) {
    uint4 x = base[w];
    const uint32_t* u = reinterpret_cast<const uint32_t*>(&x);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (Elem<T>::bytes == 4) {
        m = fmaxf(m, __uint_as_float(u[c] & 0x7fffffffu));
      } else {
        m = fmaxf(m, __uint_as_float((u[c] << 16) & 0x7fffffffu));
        m = fmaxf(m, __uint_as_float(u[c] & 0x7fff0000u));
      }
    }
  }
  m = wave_max_f(m);
  __shared__ float part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float r = part[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = fmaxf(r, part[i]);
    atomicMax(vmax_bits + s, __float_as_uint(r));
  }
}

__global__ void zero_u32_kernel(uint32_t* p, int64_t count) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0u;
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

// ---------------------------------------------------------------------------
// Cross-lane helpers (VALU only, no LDS crossbar).
// ---------------------------------------------------------------------------
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

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
// Row-pair terms.  For the 16-row tile held as fragments (lane l: row l%16,
// column quarter l/16): the float64 self dots <k,k>, <v,v> of every row and
// the cross dots <k,k'>, <v,v'> of every pair (rows 2q, 2q+1).  bf16: each
// v_dot2 gives two exact products summed in fp32, accumulated in fp64; fp32:
// fp64 FMAs.  The cross dot is split between the two partner lanes (each
// takes half of the quarter).  From them: h2 = the pair's larger diagonal
// exponent ||k||^2/sqrt(d) in base 2, rounded to float (that float is used
// wherever the pair's kappa values are scaled by exp(-h)), and lbt = log of
// the RKHS distance b (Algorithm A.1) scaled by exp(-h/2).  The
// exponentials and the log are float32 (about 1e-7 relative) on float64
// arguments; the sums are float64.
// ---------------------------------------------------------------------------
// Float64 partial dots of this lane's quarter of its row with itself (sk,
// sv) and with the partner row's quarter (ck, cv).
// bf16: each v_dot2 adds two exact products to an fp32 partial; a partial
// covers 8 elements and is then added in fp64.
template <typename T, int D>
__device__ __forceinline__ void quarter_dots_bf16(const uint4* fk, const uint4* fv, double& sk,
                                                  double& sv, double& ck, double& cv) {
  constexpr int NW = Frag<T, D>::NV * 4;
  const uint32_t* wk = reinterpret_cast<const uint32_t*>(fk);
  const uint32_t* wv = reinterpret_cast<const uint32_t*>(fv);
  sk = 0.0; sv = 0.0; ck = 0.0; cv = 0.0;
#pragma unroll
  for (int c = 0; c < NW / 4; ++c) {
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t xk = wk[4 * c + q], xv = wv[4 * c + q];
      const bf16x2_t bk = __builtin_bit_cast(bf16x2_t, xk);
      const bf16x2_t bv = __builtin_bit_cast(bf16x2_t, xv);
      const bf16x2_t pk = __builtin_bit_cast(bf16x2_t, from_partner(xk));
      const bf16x2_t pv = __builtin_bit_cast(bf16x2_t, from_partner(xv));
      a0 = __builtin_amdgcn_fdot2_f32_bf16(bk, bk, a0, false);
      a1 = __builtin_amdgcn_fdot2_f32_bf16(bv, bv, a1, false);
      a2 = __builtin_amdgcn_fdot2_f32_bf16(bk, pk, a2, false);
      a3 = __builtin_amdgcn_fdot2_f32_bf16(bv, pv, a3, false);
    }
    sk += (double)a0;
    sv += (double)a1;
    ck += (double)a2;
    cv += (double)a3;
  }
}

// fp32: exact products in fp64.
template <typename T, int D>
__device__ __forceinline__ void quarter_dots_f32(const uint4* fk, const uint4* fv, double& sk,
                                                 double& sv, double& ck, double& cv) {
  constexpr int NW = Frag<T, D>::NV * 4;
  const uint32_t* wk = reinterpret_cast<const uint32_t*>(fk);
  const uint32_t* wv = reinterpret_cast<const uint32_t*>(fv);
  sk = 0.0; sv = 0.0; ck = 0.0; cv = 0.0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const double xk = (double)__uint_as_float(wk[w]), xv = (double)__uint_as_float(wv[w]);
    const double pk = (double)__uint_as_float(from_partner(wk[w]));
    const double pv = (double)__uint_as_float(from_partner(wv[w]));
    sk = fma(xk, xk, sk);
    sv = fma(xv, xv, sv);
    ck = fma(xk, pk, ck);
    cv = fma(xv, pv, cv);
  }
}

// Row-pair terms of the 16-row tile held as fragments: h2f = the pair's
// larger diagonal exponent ||k||^2/sqrt(d) in base 2, rounded to float (that
// float is used wherever the pair's kappa values are scaled by exp(-h)), and
// lbt = log of the RKHS distance b (Algorithm A.1) scaled by exp(-h/2).
// Dots in float64; the exponentials and the log are float32 (about 1e-7
// relative) on float64 arguments; the sums are float64.
template <typename T, int D>
__device__ __forceinline__ void frag_pair_terms(const uint4* fk, const uint4* fv, double vm2d,
                                                double inv_sqrt_d, float& h2f, float& lbt) {
  double sk, sv, ck, cv;
  if (Elem<T>::bytes == 2)
    quarter_dots_bf16<T, D>(fk, fv, sk, sv, ck, cv);
  else
    quarter_dots_f32<T, D>(fk, fv, sk, sv, ck, cv);
  sk = sum_quarters(sk);
  sv = sum_quarters(sv);
  ck = sum_quarters(ck);
  cv = sum_quarters(cv);
  const double skp = from_partner(sk), svp = from_partner(sv);
  const double ex = sk * inv_sqrt_d, exp_ = skp * inv_sqrt_d, exx = ck * inv_sqrt_d;
  const double h = ex > exp_ ? ex : exp_;
  h2f = (float)(h * kLog2e);
  const double h2 = (double)h2f;
  const double t1 = (double)__builtin_amdgcn_exp2f((float)(ex * kLog2e - h2)) * (sv + vm2d);
  const double t2 = (double)__builtin_amdgcn_exp2f((float)(exp_ * kLog2e - h2)) * (svp + vm2d);
  const double t3 = (double)__builtin_amdgcn_exp2f((float)(exx * kLog2e - h2)) * (cv + vm2d);
  const double bt2 = t1 + t2 - 2.0 * t3;
  if (bt2 >= 1e-30)
    lbt = (float)(0.5 * kLn2) * __builtin_amdgcn_logf((float)bt2);
  else
    lbt = bt2 > 0.0 ? (float)(0.5 * log(bt2)) : -INFINITY;
}

// ---------------------------------------------------------------------------
// One Halve round: KH(1/2) (App. A, Algorithm A.1) on every bucket.
//
// One workgroup per bucket of N rows y_0..y_{N-1} (pair p = (y_{2p}, y_{2p+1})).
// The literal score alpha_p = sum_{S2} f_p - sum_{S1} f_p is kept per pair and
// grown incrementally: once pair i is decided with sign sgn_i (+1 kept the
// first element, -1 swapped), every later pair p receives
//     sgn_i E(i,p),  E(i,p) = k(y'_i,y_p) - k(y_i,y_p) - k(y'_i,y'_p) + k(y_i,y'_p),
// which is the same sum, reordered.  Pairs are processed in blocks of BP:
//   1. the E(i,p) of the block's own pairs come from one MFMA Gram tile;
//   2. wave 0 takes the BP decisions one after the other (ballot on
//      alpha < a (1 - 2u), the exact form of "u < min(1, (1 - alpha/a)_+/2)");
//   3. all waves add the block's contribution to every later pair: a
//      [block rows] x [later rows] Gram tile on MFMA, exp, signed reduction.
// The bucket's row indices are staged in LDS; the next column tiles are
// loaded while the current one is used; the float64 pair terms of every pair
// are formed the first time its rows are loaded (block 0's pass).
// Scaling: all kappa values feeding pair p are multiplied by exp(-h_p), h_p =
// the larger of the pair's two diagonal exponents ||k||^2/sqrt d.  This keeps
// fp32 exps in range (kappa_att overflows fp32 for large keys); the decision
// only depends on alpha/a, which the common factor leaves unchanged.  alpha
// accumulates in float64.
// ---------------------------------------------------------------------------
#ifndef HALVE_PF
#define HALVE_PF 2
#endif
#ifndef HALVE_WPE
#define HALVE_WPE 1
#endif
template <typename T, int D, int RT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(HALVE_WPE)))
void halve_kernel(HalveArgs a) {
  constexpr int NV = Frag<T, D>::NV;
  constexpr int BR = 16 * RT;  // rows per block
  constexpr int BP = BR / 2;   // pairs per block
  constexpr int ES = BP + 1;   // padded row stride of the E tile
  static_assert(BP <= 64, "decisions use one wavefront");

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int m16 = lane & 15;
  const int g = lane >> 4;

  const int64_t s = (int64_t)blockIdx.x / a.G;
  const int64_t t = (int64_t)blockIdx.x % a.G;
  const int N = a.N;
  const int P = N >> 1;
  const T* K = reinterpret_cast<const T*>(a.K) + s * a.n * D;
  const T* V = reinterpret_cast<const T*>(a.V) + s * a.n * D;
  const int32_t* rows_in = a.idx_in ? a.idx_in + s * a.n_r + t * (int64_t)N : nullptr;
  const int64_t row_base = t * (int64_t)N;
  const float* Ub = a.U + s * a.u_slice + a.u_off + t * (int64_t)P;
  uint8_t* trace = a.trace ? a.trace + s * a.u_slice + a.u_off + t * (int64_t)P : nullptr;
  int32_t* out = a.idx_out + s * (a.n_r >> 1) + t * (int64_t)P;

  extern __shared__ __align__(16) unsigned char smem[];
  double* s_alpha = reinterpret_cast<double*>(smem);
  float* s_lbt = reinterpret_cast<float*>(s_alpha + P);
  float* s_h2 = s_lbt + P;
  float* s_E = s_h2 + P;
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(s_E + BP * ES);
  int32_t* s_rows = reinterpret_cast<int32_t*>(s_mask + 4);

  const float vmax = __uint_as_float(a.vmax_bits[s]);
  const float vm2f = vmax * vmax;
  const double vm2d = (double)vmax * (double)vmax;
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  const float c2 = (float)(kLog2e * inv_sqrt_d);

  for (int j = threadIdx.x; j < N; j += 64 * WAVES)
    s_rows[j] = rows_in ? rows_in[j] : (int32_t)(row_base + j);
  for (int p = threadIdx.x; p < P; p += 64 * WAVES) s_alpha[p] = 0.0;
  __syncthreads();

  const int nblk = (N + BR - 1) / BR;
  uint4 Ak[RT][NV], Av[RT][NV];
  {
    const int nrows = min(BR, N);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int jl = rt * 16 + m16;
      const bool valid = jl < nrows;
      const int64_t r = valid ? s_rows[jl] : 0;
      load_frag<T, D>(K, r, g, valid, Ak[rt]);
      load_frag<T, D>(V, r, g, valid, Av[rt]);
    }
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      if (rt % WAVES != wave) continue;
      float h2f, lbt;
      frag_pair_terms<T, D>(Ak[rt], Av[rt], vm2d, inv_sqrt_d, h2f, lbt);
      const int jl = rt * 16 + m16;
      if (g == 0 && jl < nrows && (jl & 1) == 0) {
        s_h2[jl >> 1] = h2f;
        s_lbt[jl >> 1] = lbt;
      }
    }
  }
  // v_max enters the V Gram as one extra k-chunk: B holds v_max in slot 0 of
  // lane group 0, A holds +-v_max (the row's sign) there.
  uint4 Baug = make_uint4(0, 0, 0, 0);
  if (g == 0) Baug.x = Elem<T>::bytes == 2 ? (__float_as_uint(vmax) >> 16) : __float_as_uint(vmax);
  __syncthreads();

  double carry = -INFINITY;  // log b_max over the pairs already decided (wave 0)
  for (int blk = 0; blk < nblk; ++blk) {
    const int rows0 = blk * BR;
    const int nrows = min(BR, N - rows0);
    const int npb = nrows >> 1;
    const bool has_next = blk + 1 < nblk;
    const float u_blk = (wave == 0 && lane < npb) ? Ub[blk * BP + lane] : 0.5f;

    // ---- 1. E(i,p) for the block's own pairs. ----
#pragma unroll
    for (int rtm = 0; rtm < RT; ++rtm)
#pragma unroll
      for (int rtn = rtm; rtn < RT; ++rtn) {
        if ((rtm * RT + rtn) % WAVES != wave) continue;
        floatx4_t gk = {0.f, 0.f, 0.f, 0.f}, gv = {0.f, 0.f, 0.f, 0.f};
        gk = mma_rows<T, D>(Ak[rtm], Ak[rtn], gk);
        gv = mma_rows<T, D>(Av[rtm], Av[rtn], gv);
        const int tl = rtn * 16 + m16;  // column row (block-local)
        const float h2_in = s_h2[min(blk * BP + (tl >> 1), P - 1)];
        const float h2 = tl < nrows ? h2_in : 0.0f;
        float kap[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          kap[i] = __builtin_amdgcn_exp2f(fminf(gk[i] * c2 - h2, kExpClamp)) * (gv[i] + vm2f);
        const float F0 = kap[1] - kap[0];
        const float F1 = kap[3] - kap[2];
        const float F0p = from_partner(F0);
        const float F1p = from_partner(F1);
        if ((m16 & 1) == 0) {
          const int i0 = rtm * 8 + 2 * g;
          const int p = rtn * 8 + (m16 >> 1);
          s_E[i0 * ES + p] = F0 - F0p;
          s_E[(i0 + 1) * ES + p] = F1 - F1p;
        }
      }
    __syncthreads();

    // ---- 2. Sequential decisions (wave 0). ----
    if (wave == 0) {
      const int p = lane;
      const bool active = p < npb;
      const int gp = blk * BP + p;
      const int gpc = min(gp, P - 1);
      const double alpha_in = s_alpha[gpc];
      const float lbt_in = s_lbt[gpc];
      const float h2_in = s_h2[gpc];
      double alpha = active ? alpha_in : 0.0;
      const float lbtf = active ? lbt_in : -INFINITY;
      const float h2f = active ? h2_in : 0.0f;
      const double half_h = (double)h2f * (0.5 * kLn2);
      // running maximum of log b over this block's pairs (pair order), then
      // combined with the maximum over all earlier blocks
      const double pm = prefix_max32(active ? (double)lbtf + half_h : -INFINITY, lane);
      const double lbmax = fmax(carry, pm);
      double thr;
      if (!(lbtf > -INFINITY) || !(lbmax > -INFINITY)) {
        thr = (u_blk < 0.5f) ? INFINITY : -INFINITY;  // a = 0: p = 1/2
      } else {
        thr = exp_fast((double)lbtf + lbmax + a.log_c - half_h) * (1.0 - 2.0 * (double)u_blk);
      }
      // unconditional LDS reads (in bounds for every lane), masked afterwards
      const int pc = p < BP ? p : BP - 1;
      float ecol[BP];
#pragma unroll
      for (int i = 0; i < BP; ++i) ecol[i] = s_E[i * ES + pc];
#pragma unroll
      for (int i = 0; i < BP; ++i) ecol[i] = (active && p > i) ? ecol[i] : 0.0f;
      uint64_t smask = 0;
#pragma unroll
      for (int i = 0; i < BP; ++i) {
        if (i < npb) {
          const uint64_t bal = __ballot(alpha < thr);
          const uint64_t si = (bal >> i) & 1ull;
          smask |= si << i;
          const double e = (double)ecol[i];
          alpha += si ? -e : e;
        }
      }
      carry = __shfl(lbmax, npb - 1);
      if (active) {
        const uint32_t bit = (uint32_t)((smask >> p) & 1ull);
        out[gp] = s_rows[rows0 + 2 * p + (int)bit];
        if (trace) trace[gp] = (uint8_t)bit;
      }
      if (lane == 0) {
        s_mask[0] = (uint32_t)smask;
        s_mask[1] = (uint32_t)(smask >> 32);
      }
    }
    __syncthreads();
    if (!has_next) break;

    // ---- 3. Contribution of this block to every later pair. ----
    const uint64_t smask = (uint64_t)s_mask[0] | ((uint64_t)s_mask[1] << 32);
    // Row weights: +1 for the element that went to coreset 2, -1 for coreset 1.
    // V rows and their v_max slot carry the sign.
    uint4 Aaug[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int jl = rt * 16 + m16;
      const uint32_t bit = (uint32_t)((smask >> (jl >> 1)) & 1ull);
      const bool neg = (bit != 0) == ((jl & 1) != 0);
      const bool live = jl < nrows;
      if (live && neg) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          Av[rt][v].x ^= Elem<T>::sign_mask;
          Av[rt][v].y ^= Elem<T>::sign_mask;
          Av[rt][v].z ^= Elem<T>::sign_mask;
          Av[rt][v].w ^= Elem<T>::sign_mask;
        }
      }
      Aaug[rt] = make_uint4(0, 0, 0, 0);
      if (live) Aaug[rt].x = Baug.x ^ (neg ? (Elem<T>::bytes == 2 ? 0x8000u : 0x80000000u) : 0u);
    }
    const int later0 = rows0 + BR;
    const int ntiles = (N - later0 + 15) >> 4;
    // Ring of PF column tiles in flight (tile ct + u * WAVES sits in slot u).
    constexpr int PF = HALVE_PF;
    uint4 Bk[PF][NV], Bv[PF][NV];
#pragma unroll
    for (int u = 0; u < PF; ++u) {
      const int ct = wave + u * WAVES;
      const int64_t r = s_rows[min(later0 + ct * 16 + m16, N - 1)];
      load_frag<T, D>(K, r, g, true, Bk[u]);
      load_frag<T, D>(V, r, g, true, Bv[u]);
    }
    for (int ct0 = wave; ct0 < ntiles; ct0 += PF * WAVES) {
#pragma unroll
      for (int u = 0; u < PF; ++u) {
        const int ct = ct0 + u * WAVES;
        if (ct >= ntiles) break;
        const int tl = later0 + ct * 16 + m16;
        const bool valid = tl < N;
        float h2;
        if (blk == 0) {  // first time these rows are loaded: their pair terms
          float lbt;
          frag_pair_terms<T, D>(Bk[u], Bv[u], vm2d, inv_sqrt_d, h2, lbt);
          if (g == 0 && valid && (tl & 1) == 0) {
            s_h2[tl >> 1] = h2;
            s_lbt[tl >> 1] = lbt;
          }
          if (!valid) h2 = 0.0f;
        } else {
          const float h2_in = s_h2[min(tl, N - 1) >> 1];
          h2 = valid ? h2_in : 0.0f;
        }
        // 2*RT independent accumulators, k-chunk outermost, so consecutive
        // MFMAs never depend on each other.
        floatx4_t gk[RT], gv[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          gk[rt] = (floatx4_t){0.f, 0.f, 0.f, 0.f};
          gv[rt] = mma_aug<T>(Aaug[rt], Baug, (floatx4_t){0.f, 0.f, 0.f, 0.f});
        }
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            gk[rt] = mma_word<T>(Ak[rt][v], Bk[u][v], gk[rt]);
            gv[rt] = mma_word<T>(Av[rt][v], Bv[u][v], gv[rt]);
          }
        float acc = 0.0f;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc = fmaf(__builtin_amdgcn_exp2f(fminf(gk[rt][i] * c2 - h2, kExpClamp)), gv[rt][i], acc);
        // Refill this slot with the tile PF steps ahead.
        {
          // (rows past the bucket end load a valid row; their results are unused)
          const int nct = ct + PF * WAVES;
          const int64_t r2 = s_rows[min(later0 + nct * 16 + m16, N - 1)];
          load_frag<T, D>(K, r2, g, true, Bk[u]);
          load_frag<T, D>(V, r2, g, true, Bv[u]);
        }
        const float dt = sum_quarters(acc);
        const float dp = from_partner(dt);
        if (g == 0 && valid && (tl & 1) == 0) atomicAdd(&s_alpha[tl >> 1], (double)dt - (double)dp);
      }
    }
    // Next block's rows.
    {
      const int rows1 = rows0 + BR;
      const int nrows1 = min(BR, N - rows1);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int jl = rt * 16 + m16;
        const bool valid = jl < nrows1;
        const int64_t r = valid ? s_rows[rows1 + jl] : 0;
        load_frag<T, D>(K, r, g, valid, Ak[rt]);
        load_frag<T, D>(V, r, g, valid, Av[rt]);
      }
    }
    __syncthreads();
  }
}

// Gram of rows [0,16) against rows [16,32) through the fragment path used by
// the halving kernel (lane-layout self-check).
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

#ifndef HALVE_RT128
#define HALVE_RT128 4
#endif
template <typename T, int D>
constexpr int rt_for() {
  return (Elem<T>::bytes == 4 && D == 128) ? 2 : (D == 128 ? HALVE_RT128 : 4);
}

template <typename T, int D, int WAVES>
hipError_t launch_halve_t(const HalveArgs& a, size_t lds, hipStream_t st) {
  constexpr int RT = rt_for<T, D>();
  auto kern = halve_kernel<T, D, RT, WAVES>;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  dim3 grid((unsigned)(a.S * a.G)), block(64 * WAVES);
  hipLaunchKernelGGL(kern, grid, block, lds, st, a);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_halve_d(const HalveArgs& a, size_t lds, hipStream_t st) {
  // Enough waves in flight for the 256 CUs x 4 SIMDs x HALVE_WPE waves, at
  // most eight per bucket.
  const int64_t slots = 1024 * HALVE_WPE;  // one wave per SIMD per unit
  const int64_t buckets = a.S * (int64_t)a.G;
  if (buckets >= slots || a.N <= 64) return launch_halve_t<T, D, 1>(a, lds, st);
  if (buckets * 2 >= slots) return launch_halve_t<T, D, 2>(a, lds, st);
  if (buckets * 4 >= slots || HALVE_WPE == 1) return launch_halve_t<T, D, 4>(a, lds, st);
  return launch_halve_t<T, D, 8>(a, lds, st);
}

template <typename T>
hipError_t launch_halve_dt(int64_t d, const HalveArgs& a, size_t lds, hipStream_t st) {
  switch (d) {
    case 32: return launch_halve_d<T, 32>(a, lds, st);
    case 64: return launch_halve_d<T, 64>(a, lds, st);
    case 128: return launch_halve_d<T, 128>(a, lds, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t halve_lds_bytes(int dtype, int64_t d, int32_t N) {
  const int RT = (dtype == 0 && d == 128) ? 2 : (d == 128 ? HALVE_RT128 : 4);
  const int BP = 8 * RT;
  const size_t P = (size_t)N / 2;
  // alpha (f64), lbt, h2 per pair; E tile; mask words; row indices
  return P * (8 + 4 + 4) + (size_t)BP * (BP + 1) * 4 + 16 + (size_t)N * 4;
}

hipError_t launch_halve(int dtype, int64_t d, const HalveArgs& a, hipStream_t st) {
  const size_t lds = halve_lds_bytes(dtype, d, a.N);
  if (dtype == 0) return launch_halve_dt<float>(d, a, lds, st);
  return launch_halve_dt<bf16_t>(d, a, lds, st);
}

hipError_t launch_vmax(int dtype, const void* V, int64_t S, int64_t n, int64_t d,
                       uint32_t* vmax_bits, hipStream_t st) {
  hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)((S + 255) / 256)), dim3(256), 0, st,
                     vmax_bits, S);
  const int64_t bytes = dtype == 0 ? 4 : 2;
  const int64_t words = n * d * bytes / 16;
  const int64_t per_block = 16384;  // 256 KiB of V per workgroup
  const int64_t chunks = (words + per_block - 1) / per_block;
  dim3 grid((unsigned)chunks, (unsigned)S);
  if (dtype == 0)
    hipLaunchKernelGGL(vmax_kernel<float>, grid, dim3(256), 0, st, (const float*)V, words,
                       per_block, vmax_bits);
  else
    hipLaunchKernelGGL(vmax_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)V, words,
                       per_block, vmax_bits);
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
