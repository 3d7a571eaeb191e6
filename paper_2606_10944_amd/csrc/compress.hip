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

__device__ __forceinline__ float wave_max(float v) {
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
  m = wave_max(m);
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
// Scaling: all kappa values feeding pair p are multiplied by exp(-h_p), h_p =
// the larger of the pair's two diagonal exponents ||k||^2/sqrt d.  This keeps
// fp32 exps in range (kappa_att overflows fp32 for large keys); the decision
// only depends on alpha/a, which the common factor leaves unchanged.  The
// pair terms b_p (RKHS distance) are computed in float64 from the inputs;
// alpha accumulates in float64.
// ---------------------------------------------------------------------------
template <typename T, int D, int RT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void halve_kernel(HalveArgs a) {
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

  const float vmax = __uint_as_float(a.vmax_bits[s]);
  const float vm2f = vmax * vmax;
  const double vm2d = (double)vmax * (double)vmax;
  const double inv_sqrt_d = 1.0 / sqrt((double)D);
  const float c2 = (float)(kLog2e * inv_sqrt_d);

  auto row_of = [&](int j) -> int64_t { return rows_in ? (int64_t)rows_in[j] : row_base + j; };

  // ---- Phase A: per-pair terms (float64 dots of the raw inputs). ----
  for (int tile = wave; tile * 16 < N; tile += WAVES) {
    const int j = tile * 16 + m16;
    const bool valid = j < N;
    const int64_t r = valid ? row_of(j) : 0;
    const int64_t rp = valid ? row_of(j ^ 1) : 0;
    uint4 kx[NV], kp[NV], vx[NV], vp[NV];
    load_frag<T, D>(K, r, g, valid, kx);
    load_frag<T, D>(K, rp, g, valid, kp);
    load_frag<T, D>(V, r, g, valid, vx);
    load_frag<T, D>(V, rp, g, valid, vp);
    double sk = 0.0, ck = 0.0, sv = 0.0, cv = 0.0;
#pragma unroll
    for (int e = 0; e < D / 4; ++e) {
      const double x = elem_to_float<T>(kx, e), y = elem_to_float<T>(kp, e);
      const double z = elem_to_float<T>(vx, e), w = elem_to_float<T>(vp, e);
      sk += x * x;
      ck += x * y;
      sv += z * z;
      cv += z * w;
    }
    sk += __shfl_xor(sk, 16);
    ck += __shfl_xor(ck, 16);
    sv += __shfl_xor(sv, 16);
    cv += __shfl_xor(cv, 16);
    sk += __shfl_xor(sk, 32);
    ck += __shfl_xor(ck, 32);
    sv += __shfl_xor(sv, 32);
    cv += __shfl_xor(cv, 32);
    const double skp = __shfl_xor(sk, 1);
    const double svp = __shfl_xor(sv, 1);
    if (g == 0 && valid && (j & 1) == 0) {
      const int p = j >> 1;
      const double ex = sk * inv_sqrt_d, exp_ = skp * inv_sqrt_d, exx = ck * inv_sqrt_d;
      const double h = ex > exp_ ? ex : exp_;
      const float h2f = (float)(h * kLog2e);
      const double hu = (double)h2f * kLn2;
      const double bt2 = exp(ex - hu) * (sv + vm2d) + exp(exp_ - hu) * (svp + vm2d) -
                         2.0 * exp(exx - hu) * (cv + vm2d);
      s_h2[p] = h2f;
      s_lbt[p] = bt2 > 0.0 ? (float)(0.5 * log(bt2)) : -INFINITY;
      s_alpha[p] = 0.0;
    }
  }
  __syncthreads();

  double carry = -INFINITY;  // log b_max over the pairs already decided (wave 0)
  const int nblk = (N + BR - 1) / BR;
  for (int blk = 0; blk < nblk; ++blk) {
    const int rows0 = blk * BR;
    const int nrows = min(BR, N - rows0);
    const int npb = nrows >> 1;

    uint4 Ak[RT][NV], Av[RT][NV];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int jl = rt * 16 + m16;
      const bool valid = jl < nrows;
      const int64_t r = valid ? row_of(rows0 + jl) : 0;
      load_frag<T, D>(K, r, g, valid, Ak[rt]);
      load_frag<T, D>(V, r, g, valid, Av[rt]);
    }

    // ---- 1. E(i,p) for the block's own pairs. ----
    for (int tid = wave; tid < RT * RT; tid += WAVES) {
      const int rtm = tid / RT, rtn = tid % RT;
      if (rtm > rtn) continue;
      floatx4_t gk = {0.f, 0.f, 0.f, 0.f}, gv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        if (rt == rtm) {
#pragma unroll
          for (int rn = 0; rn < RT; ++rn)
            if (rn == rtn) {
              gk = mma_rows<T, D>(Ak[rt], Ak[rn], gk);
              gv = mma_rows<T, D>(Av[rt], Av[rn], gv);
            }
        }
      const int tl = rtn * 16 + m16;  // column row (block-local)
      const float h2 = tl < nrows ? s_h2[blk * BP + (tl >> 1)] : 0.0f;
      float kap[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        kap[i] = __builtin_amdgcn_exp2f(fminf(gk[i] * c2 - h2, kExpClamp)) * (gv[i] + vm2f);
      const float F0 = kap[1] - kap[0];
      const float F1 = kap[3] - kap[2];
      const float F0p = __shfl_xor(F0, 1);
      const float F1p = __shfl_xor(F1, 1);
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
      double alpha = active ? s_alpha[gp] : 0.0;
      const float lbtf = active ? s_lbt[gp] : -INFINITY;
      const float h2f = active ? s_h2[gp] : 0.0f;
      const double half_h = (double)h2f * (0.5 * kLn2);
      double pm = active ? (double)lbtf + half_h : -INFINITY;  // log b_p
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const double o = __shfl_up(pm, off);
        if (lane >= off) pm = fmax(pm, o);
      }
      const double lbmax = fmax(carry, pm);
      const float u = active ? Ub[gp] : 0.5f;
      double thr;
      if (!(lbtf > -INFINITY) || !(lbmax > -INFINITY)) {
        thr = (u < 0.5f) ? INFINITY : -INFINITY;  // a = 0: p = 1/2
      } else {
        thr = exp((double)lbtf + lbmax + a.log_c - half_h) * (1.0 - 2.0 * (double)u);
      }
      float ecol[BP];
#pragma unroll
      for (int i = 0; i < BP; ++i) ecol[i] = (active && p > i) ? s_E[i * ES + p] : 0.0f;
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
        out[gp] = (int32_t)(bit ? row_of(rows0 + 2 * p + 1) : row_of(rows0 + 2 * p));
        if (trace) trace[gp] = (uint8_t)bit;
      }
      if (lane == 0) {
        s_mask[0] = (uint32_t)smask;
        s_mask[1] = (uint32_t)(smask >> 32);
      }
    }
    __syncthreads();
    if (blk == nblk - 1) break;

    // ---- 3. Contribution of this block to every later pair. ----
    const uint64_t smask = (uint64_t)s_mask[0] | ((uint64_t)s_mask[1] << 32);
    // Row weights: +1 for the element that went to coreset 2, -1 for coreset 1.
    float cw[RT][4];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int jl = rt * 16 + m16;
      const uint32_t bit = (uint32_t)((smask >> (jl >> 1)) & 1ull);
      const bool neg = (bit != 0) == ((jl & 1) != 0);
      if (jl < nrows && neg) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          Av[rt][v].x ^= Elem<T>::sign_mask;
          Av[rt][v].y ^= Elem<T>::sign_mask;
          Av[rt][v].z ^= Elem<T>::sign_mask;
          Av[rt][v].w ^= Elem<T>::sign_mask;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int jr = rt * 16 + 4 * g + i;
        const uint32_t b2 = (uint32_t)((smask >> (jr >> 1)) & 1ull);
        const bool n2 = (b2 != 0) == ((jr & 1) != 0);
        cw[rt][i] = jr < nrows ? (n2 ? -vm2f : vm2f) : 0.0f;
      }
    }
    const int later0 = rows0 + BR;
    const int ntiles = (N - later0 + 15) >> 4;
    for (int ct = wave; ct < ntiles; ct += WAVES) {
      const int tl = later0 + ct * 16 + m16;
      const bool valid = tl < N;
      const int64_t r = valid ? row_of(tl) : 0;
      uint4 Bk[NV], Bv[NV];
      load_frag<T, D>(K, r, g, valid, Bk);
      load_frag<T, D>(V, r, g, valid, Bv);
      const float h2 = valid ? s_h2[tl >> 1] : 0.0f;
      float acc = 0.0f;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        floatx4_t gk = {0.f, 0.f, 0.f, 0.f}, gv = {0.f, 0.f, 0.f, 0.f};
        gk = mma_rows<T, D>(Ak[rt], Bk, gk);
        gv = mma_rows<T, D>(Av[rt], Bv, gv);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          acc = fmaf(__builtin_amdgcn_exp2f(fminf(gk[i] * c2 - h2, kExpClamp)), gv[i] + cw[rt][i], acc);
      }
      double dd = (double)acc;
      dd += __shfl_xor(dd, 16);
      dd += __shfl_xor(dd, 32);
      const double dp = __shfl_xor(dd, 1);
      if (g == 0 && valid && (tl & 1) == 0) s_alpha[tl >> 1] += dd - dp;
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

template <typename T, int D>
constexpr int rt_for() {
  return (Elem<T>::bytes == 4 && D == 128) ? 2 : 4;
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
  if (a.N <= 256) return launch_halve_t<T, D, 1>(a, lds, st);
  if (a.N <= 512) return launch_halve_t<T, D, 2>(a, lds, st);
  // Eight waves only where the register budget (256 per lane) holds the block.
  constexpr bool eight = (Elem<T>::bytes == 2 && D <= 64) || D <= 32;
  if (a.N <= 1024 || !eight) return launch_halve_t<T, D, 4>(a, lds, st);
  return launch_halve_t<T, D, eight ? 8 : 4>(a, lds, st);
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
  const int RT = (dtype == 0 && d == 128) ? 2 : 4;
  const int BP = 8 * RT;
  const size_t P = (size_t)N / 2;
  return P * (8 + 4 + 4) + (size_t)BP * (BP + 1) * 4 + 16;
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
