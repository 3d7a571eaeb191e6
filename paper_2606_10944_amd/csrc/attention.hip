// Coreset attention on gfx950: every query of a slice attends over the n_out
// rows idx[s, :] of that slice's K/V (Sec. 2.1 eq. unmaskedatt on the
// coreset; eq. def:att_approx with equal weights, which cancel).  The
// weighted variant (W) gives key j the weight exp(logw[s, j]): its raw score
// <q, k_j> gets the bias sqrt(d) * logw[s, j], staged in LDS beside the keys
// (a key past n_out or of weight 0 has bias -inf, which also masks it).
//
// One workgroup = 4 waves = 128 queries of one slice.  The coreset is walked
// in chunks of 64 keys staged in LDS (gathered through idx); scores S^T =
// K_I Q^T come from 16x16 MFMA tiles (keys x queries), the softmax is online
// in float32, and O^T += V_I^T P^T reuses the score tile's register layout as
// the B operand.  For bf16 inputs the weights P (float32) enter the bf16 P.V
// MFMA as two terms, P = hi + lo with hi = bf16(P), lo = bf16(P - hi), so the
// product keeps about 16 significant bits of P instead of 8.
#include <math.h>

#include "common.hpp"
#include "launch.hpp"

namespace thin {

namespace {

constexpr int KC = 64;   // keys per chunk
constexpr int QT = 2;    // 16-query tiles per wave
constexpr int WAVES = 4;
constexpr int QPB = 16 * QT * WAVES;  // queries per workgroup
// The prefill kernel takes the same 128 queries per workgroup as 8 waves of
// one 16-query tile: half the registers per wave (128, four waves per SIMD,
// two workgroups per CU), so a chunk's gathers, barriers and arithmetic of
// one workgroup overlap the other's (65536 points x 32 slices: 8.19 -> 5.76
// ms against 4 waves of two tiles).
constexpr int PF_QT = 1;
constexpr int PF_WAVES = 8;
static_assert(16 * PF_QT * PF_WAVES == QPB, "prefill tiles of QPB points");
constexpr double kLog2e = 1.44269504088896340736;

template <typename T, int D>
struct AttnLds {
  // K chunk, row-major, padded by 16 bytes per row.
  static constexpr int k_stride = D * Elem<T>::bytes + 16;
  // V chunk: bf16 is stored transposed [D][KC] (+8 elements pad), fp32 row-major.
  static constexpr int v_stride = Elem<T>::bytes == 2 ? (KC + 8) * 2 : D * 4 + 16;
  static constexpr int v_rows = Elem<T>::bytes == 2 ? D : KC;
  static constexpr int bytes = KC * k_stride + v_rows * v_stride + KC * 4;
};

template <typename TO>
__device__ __forceinline__ void store4(TO* p, float a, float b, float c, float d);

template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  const b2 lo = {(__bf16)a, (__bf16)b}, hi = {(__bf16)c, (__bf16)d};
  *reinterpret_cast<uint2*>(p) = make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
}

template <typename T, int D, typename TO, bool W>
__global__ __launch_bounds__(64 * WAVES) void coreset_attn_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const int32_t* __restrict__ idx, const float* __restrict__ logw, int64_t n, int64_t n_q,
    int n_out, TO* __restrict__ O) {
  constexpr int NV = Frag<T, D>::NV;
  constexpr bool BF = Elem<T>::bytes == 2;
  using L = AttnLds<T, D>;
  __shared__ __align__(16) unsigned char lds[L::bytes];
  unsigned char* sK = lds;
  unsigned char* sV = lds + KC * L::k_stride;
  float* sB = reinterpret_cast<float*>(sV + L::v_rows * L::v_stride);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t s = blockIdx.y;
  const int64_t q0 = (int64_t)blockIdx.x * QPB + wave * 16 * QT;
  const float* Ws = W ? logw + s * (int64_t)n_out : nullptr;
  const float sqrt_d = (float)sqrt((double)D);
  const T* Ks = K + s * n * D;
  const T* Vs = V + s * n * D;
  const int32_t* Is = idx + s * (int64_t)n_out;
  const float c2 = (float)(kLog2e / sqrt((double)D));

  uint4 Bq[QT][NV];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int64_t q = q0 + qt * 16 + m16;
    load_frag<T, D>(Q + s * n_q * D, q, g, q < n_q, Bq[qt]);
  }

  float mrun[QT], lrun[QT];
  floatx4_t acc[QT][D / 16];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    mrun[qt] = -INFINITY;
    lrun[qt] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[qt][dt] = (floatx4_t){0.f, 0.f, 0.f, 0.f};
  }

  constexpr int WPR = D * Elem<T>::bytes / 16;  // 16-byte words per row
  for (int c0 = 0; c0 < n_out; c0 += KC) {
    const int kc = min(KC, n_out - c0);
    __syncthreads();
    if (W && threadIdx.x < KC)
      sB[threadIdx.x] = (int)threadIdx.x < kc ? Ws[c0 + threadIdx.x] * sqrt_d : -INFINITY;
    for (int w = threadIdx.x; w < KC * WPR; w += 64 * WAVES) {
      const int key = w / WPR, wi = w % WPR;
      uint4 kw = make_uint4(0, 0, 0, 0), vw = make_uint4(0, 0, 0, 0);
      if (key < kc) {
        int64_t r = Is[c0 + key];
        r = r < 0 ? 0 : (r >= n ? n - 1 : r);
        kw = reinterpret_cast<const uint4*>(Ks + r * D)[wi];
        vw = reinterpret_cast<const uint4*>(Vs + r * D)[wi];
      }
      *reinterpret_cast<uint4*>(sK + key * L::k_stride + wi * 16) = kw;
      if (BF) {
        const uint16_t* e = reinterpret_cast<const uint16_t*>(&vw);
#pragma unroll
        for (int j = 0; j < 8; ++j)
          *reinterpret_cast<uint16_t*>(sV + (wi * 8 + j) * L::v_stride + key * 2) = e[j];
      } else {
        *reinterpret_cast<uint4*>(sV + key * L::v_stride + wi * 16) = vw;
      }
    }
    __syncthreads();

    uint4 Ak[4][NV];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      const uint4* p = reinterpret_cast<const uint4*>(sK + (kt * 16 + m16) * L::k_stride);
#pragma unroll
      for (int v = 0; v < NV; ++v) Ak[kt][v] = p[4 * v + g];
    }

#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float sc[4][4];
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        floatx4_t z = {0.f, 0.f, 0.f, 0.f};
        z = mma_rows<T, D>(Ak[kt], Bq[qt], z);
        if (W) {
          const float4 b = *reinterpret_cast<const float4*>(sB + kt * 16 + 4 * g);
          z[0] += b.x; z[1] += b.y; z[2] += b.z; z[3] += b.w;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kt * 16 + 4 * g + i;
          sc[kt][i] = W || key < kc ? z[i] : -INFINITY;
          mx = fmaxf(mx, sc[kt][i]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(mrun[qt], mx);
      const float scale = mrun[qt] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((mrun[qt] - mnew) * c2);
      mrun[qt] = mnew;
      float psum = 0.0f;
      float pr[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = sc[kt][i] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((sc[kt][i] - mnew) * c2);
          pr[kt][i] = pv;
          psum += pv;
        }
      lrun[qt] = lrun[qt] * scale + psum;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[qt][dt] *= scale;

      if (BF) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          float pv[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) pv[j] = pr[2 * c + (j >> 2)][j & 3];
          bf16x8_t bhi, blo;
          split_bf16x8(pv, bhi, blo);
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            const unsigned char* row = sV + (dt * 16 + m16) * L::v_stride;
            uint2 lo = *reinterpret_cast<const uint2*>(row + (32 * c + 4 * g) * 2);
            uint2 hi = *reinterpret_cast<const uint2*>(row + (32 * c + 16 + 4 * g) * 2);
            const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bhi, acc[qt][dt], 0, 0, 0);
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, blo, acc[qt][dt], 0, 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kt * 16 + 4 * g + i;
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) {
              const float av = *reinterpret_cast<const float*>(sV + key * L::v_stride + (dt * 16 + m16) * 4);
              acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, pr[kt][i], acc[qt][dt], 0, 0, 0);
            }
          }
      }
    }
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float l = lrun[qt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const float inv = 1.0f / l;
    const int64_t q = q0 + qt * 16 + m16;
    if (q < n_q) {
      TO* orow = O + (s * n_q + q) * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
        store4<TO>(orow + dt * 16 + 4 * g, acc[qt][dt][0] * inv, acc[qt][dt][1] * inv,
                   acc[qt][dt][2] * inv, acc[qt][dt][3] * inv);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16, coreset resident in LDS (n_out <= 16*NKT, NKT even).  One workgroup (WR waves)
// stays on one slice and walks a contiguous range of queries, 16*QTR per wave
// per step, with the next step's query fragments loaded during the current
// one; the coreset is staged once: K row-major, V transposed (each thread
// transposes an 8-key x 8-column block in registers).  Softmax is one pass
// over all keys.
// ---------------------------------------------------------------------------
// Row paddings of the staged coreset.  K fragments are read 16 bytes per lane
// from 16 rows at once: a stride of 68 words puts the rows on disjoint banks.
// V^T fragments are read 8 bytes per lane from 16 rows: a stride of 2 (mod 32)
// words keeps those disjoint too (a 16-byte pad gave two-way conflicts).
template <int D, int NKT>
struct ResLds {
  static constexpr int NK = 16 * NKT;          // padded key count
  static constexpr int k_stride = D * 2 + 16;  // bytes per K row
  static constexpr int v_stride = NK * 2 + 8;  // bytes per V^T row (8-byte aligned)
  static constexpr int bytes = NK * k_stride + D * v_stride + NK * 4;
  // P.V multiplies 32 keys at a time
  static_assert(NKT % 2 == 0, "resident coreset needs an even number of 16-key tiles");
};

__device__ __forceinline__ uint32_t pack_lo(uint32_t x, uint32_t y) { return (x & 0xffffu) | (y << 16); }
__device__ __forceinline__ uint32_t pack_hi(uint32_t x, uint32_t y) { return (x >> 16) | (y & 0xffff0000u); }

// Target of the output stores of query rows past a workgroup's range (never read).
__device__ __align__(16) float g_attn_sink[256];

template <int D, int NKT, int QTR, int WR, typename TO, bool W>
__global__ __launch_bounds__(64 * WR) void coreset_attn_res_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
    const int32_t* __restrict__ idx, const float* __restrict__ logw, int64_t n, int64_t n_q,
    int n_out, int64_t q_per_wg, TO* __restrict__ O) {
  using L = ResLds<D, NKT>;
  constexpr int NK = L::NK;
  constexpr int NV = Frag<bf16_t, D>::NV;
  extern __shared__ __align__(16) unsigned char lds[];
  unsigned char* sK = lds;
  unsigned char* sV = lds + NK * L::k_stride;
  float* sB = reinterpret_cast<float*>(sV + D * L::v_stride);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t s = blockIdx.y;
  if (W) {
    const float sqrt_d = (float)sqrt((double)D);
    for (int k = threadIdx.x; k < NK; k += 64 * WR)
      sB[k] = k < n_out ? logw[s * (int64_t)n_out + k] * sqrt_d : -INFINITY;
  }
  const bf16_t* Ks = K + s * n * D;
  const bf16_t* Vs = V + s * n * D;
  const int32_t* Is = idx + s * (int64_t)n_out;
  const float c2 = (float)(kLog2e / sqrt((double)D));

  // ---- stage the coreset ----
  constexpr int WPR = D / 8;  // 16-byte words per row
  for (int w = threadIdx.x; w < NK * WPR; w += 64 * WR) {
    const int key = w / WPR, wi = w % WPR;
    uint4 kw = make_uint4(0, 0, 0, 0);
    if (key < n_out) {
      int64_t r = Is[key];
      r = r < 0 ? 0 : (r >= n ? n - 1 : r);
      kw = reinterpret_cast<const uint4*>(Ks + r * D)[wi];
    }
    *reinterpret_cast<uint4*>(sK + key * L::k_stride + wi * 16) = kw;
  }
  for (int b = threadIdx.x; b < (NK / 8) * WPR; b += 64 * WR) {
    const int kb = b / WPR, db = b % WPR;  // keys 8kb..8kb+7, columns 8db..8db+7
    uint32_t w[8][4];
#pragma unroll
    for (int r8 = 0; r8 < 8; ++r8) {
      const int key = kb * 8 + r8;
      uint4 vw = make_uint4(0, 0, 0, 0);
      if (key < n_out) {
        int64_t r = Is[key];
        r = r < 0 ? 0 : (r >= n ? n - 1 : r);
        vw = reinterpret_cast<const uint4*>(Vs + r * D)[db];
      }
      w[r8][0] = vw.x; w[r8][1] = vw.y; w[r8][2] = vw.z; w[r8][3] = vw.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // column 8db + e: the 8 keys' values
      const int k = e >> 1;
      uint4 o;
      if ((e & 1) == 0) {
        o.x = pack_lo(w[0][k], w[1][k]); o.y = pack_lo(w[2][k], w[3][k]);
        o.z = pack_lo(w[4][k], w[5][k]); o.w = pack_lo(w[6][k], w[7][k]);
      } else {
        o.x = pack_hi(w[0][k], w[1][k]); o.y = pack_hi(w[2][k], w[3][k]);
        o.z = pack_hi(w[4][k], w[5][k]); o.w = pack_hi(w[6][k], w[7][k]);
      }
      unsigned char* dst = sV + (db * 8 + e) * L::v_stride + kb * 16;
      if constexpr (L::v_stride % 16 == 0) {
        *reinterpret_cast<uint4*>(dst) = o;
      } else {
        reinterpret_cast<uint2*>(dst)[0] = make_uint2(o.x, o.y);
        reinterpret_cast<uint2*>(dst)[1] = make_uint2(o.z, o.w);
      }
    }
  }
  __syncthreads();

  const int64_t q_begin = (int64_t)blockIdx.x * q_per_wg;
  const int64_t q_end = min(q_begin + q_per_wg, n_q);
  const bf16_t* Qs = Q + s * n_q * D;
  constexpr int QSTEP = 16 * QTR * WR;  // queries per workgroup step

  uint4 Bq[QTR][NV];
#pragma unroll
  for (int qt = 0; qt < QTR; ++qt) {
    const int64_t q = q_begin + wave * 16 * QTR + qt * 16 + m16;
    load_frag<bf16_t, D>(Qs, min(q, n_q - 1), g, true, Bq[qt]);
  }
  // The first queries are consumed here (the compiler waits for them before
  // the loop): the loop is then entered with nothing in flight, so its waits
  // (stores count in vmcnt) are for the next queries' loads only.
#pragma unroll
  for (int qt = 0; qt < QTR; ++qt)
#pragma unroll
    for (int v = 0; v < NV; ++v)
      asm volatile("" : "+v"(Bq[qt][v].x), "+v"(Bq[qt][v].y), "+v"(Bq[qt][v].z), "+v"(Bq[qt][v].w));
  for (int64_t q0 = q_begin; q0 < q_end; q0 += QSTEP) {
    const int64_t qw = q0 + wave * 16 * QTR;
    uint4 Nq[QTR][NV];
#pragma unroll
    for (int qt = 0; qt < QTR; ++qt) {
      const int64_t q = qw + QSTEP + qt * 16 + m16;
      load_frag<bf16_t, D>(Qs, min(q, n_q - 1), g, true, Nq[qt]);
    }
    // scores S^T[key][query]; the next key tile's fragment is read while the
    // current one multiplies, and no further (the scheduling barrier keeps
    // the compiler from hoisting every tile's LDS reads at once)
    floatx4_t sc[QTR][NKT];
    uint4 a[2][NV];
#pragma unroll
    for (int v = 0; v < NV; ++v)
      a[0][v] = reinterpret_cast<const uint4*>(sK + m16 * L::k_stride)[4 * v + g];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      if (kt + 1 < NKT) {
        const uint4* pk = reinterpret_cast<const uint4*>(sK + ((kt + 1) * 16 + m16) * L::k_stride);
#pragma unroll
        for (int v = 0; v < NV; ++v) a[(kt + 1) & 1][v] = pk[4 * v + g];
      }
#pragma unroll
      for (int qt = 0; qt < QTR; ++qt) {
        floatx4_t z = {0.f, 0.f, 0.f, 0.f};
        sc[qt][kt] = mma_rows<bf16_t, D>(a[kt & 1], Bq[qt], z);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    float inv_l[QTR];
    floatx4_t acc[QTR][D / 16];
#pragma unroll
    for (int qt = 0; qt < QTR; ++qt) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        if (W) {
          const float4 b = *reinterpret_cast<const float4*>(sB + kt * 16 + 4 * g);
          sc[qt][kt][0] += b.x; sc[qt][kt][1] += b.y; sc[qt][kt][2] += b.z; sc[qt][kt][3] += b.w;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kt * 16 + 4 * g + i;
          if (!W && key >= n_out) sc[qt][kt][i] = -INFINITY;
          mx = fmaxf(mx, sc[qt][kt][i]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      float l = 0.f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = __builtin_amdgcn_exp2f((sc[qt][kt][i] - mx) * c2);
          sc[qt][kt][i] = pv;
          l += pv;
        }
      l += __shfl_xor(l, 16);
      l += __shfl_xor(l, 32);
      inv_l[qt] = 1.0f / l;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[qt][dt] = (floatx4_t){0.f, 0.f, 0.f, 0.f};
    }
    // O^T += V^T P^T, 32 keys per MFMA; P = hi + lo in bf16
#pragma unroll
    for (int c = 0; c < NKT / 2; ++c) {
      bf16x8_t bhi[QTR], blo[QTR];
#pragma unroll
      for (int qt = 0; qt < QTR; ++qt) {
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[e] = sc[qt][2 * c + (e >> 2)][e & 3];
        split_bf16x8(pv, bhi[qt], blo[qt]);
      }
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const unsigned char* row = sV + (dt * 16 + m16) * L::v_stride;
        const uint2 lo = *reinterpret_cast<const uint2*>(row + (32 * c + 4 * g) * 2);
        const uint2 hi = *reinterpret_cast<const uint2*>(row + (32 * c + 16 + 4 * g) * 2);
        const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
        for (int qt = 0; qt < QTR; ++qt) {
          acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bhi[qt], acc[qt][dt], 0, 0, 0);
          acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, blo[qt], acc[qt][dt], 0, 0, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int qt = 0; qt < QTR; ++qt) {
      if constexpr (sizeof(TO) == 4) {
        // Whole 128-byte lines: for columns 32j..32j+31, lanes m16 < 8 hold
        // the first 16 (O^T tile 2j) and lanes m16 >= 8 the last 16 (tile
        // 2j+1) of rows m16 & 7 (store A) and (m16 & 7) + 8 (store B); the
        // missing halves come from lane l ^ 8 (DPP row rotation by 8).
        const bool upper = m16 >= 8;
        const int64_t qa = qw + qt * 16 + (m16 & 7), qb = qa + 8;
        float* ra = reinterpret_cast<float*>(O) + (s * n_q + qa) * D;
        float* rb = ra + 8 * D;
#pragma unroll
        for (int j = 0; j < D / 32; ++j) {
          float va[4], vb[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float a = acc[qt][2 * j][i] * inv_l[qt], b = acc[qt][2 * j + 1][i] * inv_l[qt];
            const float y = __uint_as_float((uint32_t)__builtin_amdgcn_mov_dpp(
                (int)__float_as_uint(upper ? a : b), 0x128, 0xF, 0xF, false));
            va[i] = upper ? y : a;
            vb[i] = upper ? b : y;
          }
          const int col = 32 * j + (upper ? 16 : 0) + 4 * g;
          // rows past the range store to a sink: the stores stay unconditional,
          // so the wait for the next queries' loads never covers them.  The
          // output is written once and not read here: non-temporal stores keep
          // it out of the caches, which the next kernels' reads would
          // otherwise first have to write back.
          float* da = qa < q_end ? ra + col : g_attn_sink + 4 * lane;
          float* db = qb < q_end ? rb + col : g_attn_sink + 4 * lane;
          typedef float f4_t __attribute__((ext_vector_type(4)));
          __builtin_nontemporal_store((f4_t){va[0], va[1], va[2], va[3]}, reinterpret_cast<f4_t*>(da));
          __builtin_nontemporal_store((f4_t){vb[0], vb[1], vb[2], vb[3]}, reinterpret_cast<f4_t*>(db));
        }
      } else {
        // bf16: lane (g, m16) holds columns 16 dt + 4g .. +3 of query m16.
        // Lanes g = 2h and 2h + 1 (16 apart) exchange one of two adjacent
        // tiles (one row swap per packed word), so that each stores 16
        // contiguous bytes: the even lane columns 16 dt_e + 8h .. +7, the odd
        // lane 16 dt_o + 8h .. +7; the four lanes of a query then write 64
        // contiguous bytes per tile pair, not 8-byte pieces.
        const int64_t q = qw + qt * 16 + m16;
        const bool oddrow = (g & 1) != 0;
        const int h = g >> 1;
        TO* orow = O + (s * n_q + min(q, q_end - 1)) * D;
#pragma unroll
        for (int k = 0; k < D / 32; ++k) {
          typedef __bf16 b2 __attribute__((ext_vector_type(2)));
          uint32_t ev[2], od[2];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const b2 e2 = {(__bf16)(acc[qt][2 * k][2 * j] * inv_l[qt]),
                           (__bf16)(acc[qt][2 * k][2 * j + 1] * inv_l[qt])};
            const b2 o2 = {(__bf16)(acc[qt][2 * k + 1][2 * j] * inv_l[qt]),
                           (__bf16)(acc[qt][2 * k + 1][2 * j + 1] * inv_l[qt])};
            ev[j] = __builtin_bit_cast(uint32_t, e2);
            od[j] = __builtin_bit_cast(uint32_t, o2);
          }
          // even row lanes receive the partner's even tile, odd row lanes the
          // partner's odd tile
          uint32_t got[2];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const auto r = __builtin_amdgcn_permlane16_swap(ev[j], od[j], false, false);
            got[j] = oddrow ? r[0] : r[1];
          }
          const uint4 w = oddrow ? make_uint4(got[0], got[1], od[0], od[1])
                                 : make_uint4(ev[0], ev[1], got[0], got[1]);
          if (q < q_end)
            *reinterpret_cast<uint4*>(orow + 16 * (2 * k + (oddrow ? 1 : 0)) + 8 * h) = w;
        }
      }
#pragma unroll
      for (int v = 0; v < NV; ++v) Bq[qt][v] = Nq[qt][v];
    }
  }
}

template <int D, int NKT, int QTR, int WR, typename TO, bool W>
hipError_t launch_attn_res_w(const void* Q, const void* K, const void* V, const int32_t* idx,
                             const float* logw, int64_t S, int64_t n, int64_t n_q,
                             int64_t n_out, void* O, hipStream_t st) {
  using L = ResLds<D, NKT>;
  auto kern = coreset_attn_res_kernel<D, NKT, QTR, WR, TO, W>;
  const size_t lds = L::bytes;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  constexpr int64_t QSTEP = 16 * QTR * WR;
  // about two workgroups per CU in total, whole steps of queries per workgroup
  int64_t per_slice = (512 + S - 1) / S;
  const int64_t steps = (n_q + QSTEP - 1) / QSTEP;
  if (per_slice > steps) per_slice = steps;
  if (per_slice < 1) per_slice = 1;
  const int64_t q_per_wg = ((steps + per_slice - 1) / per_slice) * QSTEP;
  const int64_t wgs = (n_q + q_per_wg - 1) / q_per_wg;
  dim3 grid((unsigned)wgs, (unsigned)S), block(64 * WR);
  hipLaunchKernelGGL(kern, grid, block, lds, st, (const bf16_t*)Q, (const bf16_t*)K,
                     (const bf16_t*)V, idx, logw, n, n_q, (int)n_out, q_per_wg, (TO*)O);
  return hipGetLastError();
}

template <int D, int NKT, int QTR, int WR, typename TO>
hipError_t launch_attn_res(const void* Q, const void* K, const void* V, const int32_t* idx,
                           const float* logw, int64_t S, int64_t n, int64_t n_q, int64_t n_out,
                           void* O, hipStream_t st) {
  if (logw)
    return launch_attn_res_w<D, NKT, QTR, WR, TO, true>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  return launch_attn_res_w<D, NKT, QTR, WR, TO, false>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
}

// 16-query tiles per wave per step and waves per workgroup of the resident kernel
#ifndef ATTN_RES_QTR
#define ATTN_RES_QTR 1
#endif
#ifndef ATTN_RES_WAVES
#define ATTN_RES_WAVES 4
#endif
// Coresets of 192 or 256 keys take over 100 KB of LDS, one workgroup per CU:
// eight waves then hide more latency than four (256 keys, d = 128: 353 -> 280 us
// on the long workload's queries).
#ifndef ATTN_RES_WAVES_BIG
#define ATTN_RES_WAVES_BIG 8
#endif

template <int D, typename TO>
hipError_t launch_attn_res_d(int64_t n_out, const void* Q, const void* K, const void* V,
                             const int32_t* idx, const float* logw, int64_t S, int64_t n,
                             int64_t n_q, void* O, hipStream_t st, bool* used) {
  *used = true;
  if (n_out <= 32) return launch_attn_res<D, 2, ATTN_RES_QTR, ATTN_RES_WAVES, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  if (n_out <= 64) return launch_attn_res<D, 4, ATTN_RES_QTR, ATTN_RES_WAVES, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  if (n_out <= 96) return launch_attn_res<D, 6, ATTN_RES_QTR, ATTN_RES_WAVES, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  if (n_out <= 128) return launch_attn_res<D, 8, ATTN_RES_QTR, ATTN_RES_WAVES, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  // (192 = n_out 128 plus 32 sinks and a 32-row window)
  if (n_out <= 192 && D <= 128) return launch_attn_res<D, 12, ATTN_RES_QTR, ATTN_RES_WAVES_BIG, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  if (n_out <= 256 && D <= 128) return launch_attn_res<D, 16, ATTN_RES_QTR, ATTN_RES_WAVES_BIG, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  *used = false;
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Masked (causal) prefill over the Express cache (Alg. 4 for every point at
// once).  One workgroup = the up to 128 points [q0, q1) of a tile of one
// slice.  Its keys are the tile's cache pieces (rows of the cache, each with
// one log-weight, piece k seen by the points vlo..vhi-1), then the causal
// candidates causal_lo .. q1-1: candidate r is seen by point p iff r == p
// (the point itself) or r was kept and c0[p] <= r < p (p's C_0), with p's
// log-weight w0[p].  C_0 starts never move back (c0 is non-decreasing in p),
// so the points of the tile that see a candidate are an interval too:
// [r, max(r + 1, first tile point whose C_0 starts after r)) if r was kept,
// else [r, r + 1).  Every key then carries one interval of the tile's points
// (offsets from q0 in [0, 128], start in bits 0-15, end in bits 16-30); a
// causal key is flagged by bit 31 and takes the point's bias.  Same
// arithmetic as coreset_attn_kernel, with per-key biases sqrt(d) * logw.
// ---------------------------------------------------------------------------
template <typename T, int D, typename TO>
__global__ __launch_bounds__(64 * PF_WAVES) __attribute__((amdgpu_waves_per_eu(4))) void prefill_attn_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V, int64_t n,
    const PrefillTile* __restrict__ tiles, const PrefillSeg* __restrict__ segs,
    const int32_t* __restrict__ c0s, const float* __restrict__ w0s,
    const uint8_t* __restrict__ kept, TO* __restrict__ O) {
  constexpr int NV = Frag<T, D>::NV;
  constexpr bool BF = Elem<T>::bytes == 2;
  using L = AttnLds<T, D>;
  __shared__ __align__(16) unsigned char lds[L::bytes];
  // a key's interval of the tile's points that see it (packed as above)
  __shared__ __align__(16) uint32_t s_vis[KC];
  __shared__ int32_t s_row[KC];
  __shared__ int64_t s_seg_end[kPrefillMaxSegs];
  __shared__ PrefillSeg s_seg[kPrefillMaxSegs];
  __shared__ int32_t s_c0[QPB];
  __shared__ float s_w0[QPB];
  unsigned char* sK = lds;
  unsigned char* sV = lds + KC * L::k_stride;
  float* sB = reinterpret_cast<float*>(sV + L::v_rows * L::v_stride);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t s = blockIdx.y;
  const PrefillTile tile = tiles[blockIdx.x];
  const int64_t q0 = tile.q0, q1 = tile.q1;
  const int nseg = min(tile.nseg, kPrefillMaxSegs);
  if ((int)threadIdx.x < nseg) s_seg[threadIdx.x] = segs[tile.seg0 + threadIdx.x];
  if ((int)threadIdx.x < QPB && q0 + threadIdx.x < q1) {
    s_c0[threadIdx.x] = c0s[q0 + threadIdx.x];
    s_w0[threadIdx.x] = w0s[q0 + threadIdx.x];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t e = 0;
    for (int k = 0; k < nseg; ++k) s_seg_end[k] = (e += s_seg[k].g.len);
  }
  __syncthreads();
  const int64_t F = nseg ? s_seg_end[nseg - 1] : 0;
  const int64_t M = F + (q1 - tile.causal_lo);
  const T* Ks = K + s * n * D;
  const T* Vs = V + s * n * D;
  const float sqrt_d = (float)sqrt((double)D);
  const float c2 = (float)(kLog2e / sqrt((double)D));
  const int64_t qw = q0 + wave * 16 * PF_QT;

  uint4 Bq[PF_QT][NV];
#pragma unroll
  for (int qt = 0; qt < PF_QT; ++qt) {
    const int64_t q = qw + qt * 16 + m16;
    load_frag<T, D>(Q + s * n * D, q, g, q < q1, Bq[qt]);
  }
  float mrun[PF_QT], lrun[PF_QT];
  floatx4_t acc[PF_QT][D / 16];
#pragma unroll
  for (int qt = 0; qt < PF_QT; ++qt) {
    mrun[qt] = -INFINITY;
    lrun[qt] = 0.0f;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) acc[qt][dt] = (floatx4_t){0.f, 0.f, 0.f, 0.f};
  }

  constexpr int WPR = D * Elem<T>::bytes / 16;
  // A chunk's keys (row, bias, visibility; one thread per key) are gathered
  // into registers one chunk ahead, so their list reads overlap the previous
  // chunk's arithmetic; they reach LDS at the top of the chunk.
  // (registers hold the raw loaded values; anything computed from them is
  // left to the commit, so that no wait for the loads precedes the compute)
  // m_vis / m_vis_nk: the key's packed visibility (a causal candidate's if
  // kept / if not kept; the list read of kept[] is only waited for at commit)
  uint32_t m_vis = 0, m_vis_nk = 0;
  int32_t m_raw = 0, m_cpos = -1;
  uint8_t m_kept = 1;
  float m_bias = -INFINITY;
  bool m_piece = false;
  auto gather_meta = [&](int64_t ck_) {
    if (threadIdx.x >= KC) return;
    const int kc_ = (int)min((int64_t)KC, M - ck_);
    const int64_t kk = ck_ + threadIdx.x;
    // points [lo, hi) as offsets in the tile, clipped to it
    auto vis = [&](int64_t lo, int64_t hi) {
      const uint32_t a = (uint32_t)min(max(lo - q0, (int64_t)0), (int64_t)QPB);
      const uint32_t b = (uint32_t)min(max(hi - q0, (int64_t)0), (int64_t)QPB);
      return a | (b << 16);
    };
    m_vis = 0;
    m_vis_nk = 0;
    m_bias = -INFINITY;
    m_piece = false;
    m_cpos = -1;
    m_raw = 0;
    m_kept = 1;
    if ((int)threadIdx.x < kc_) {
      if (kk < F) {
        // the piece holding key kk: the first k with kk < s_seg_end[k]
        // (binary search: a tile has up to kPrefillMaxSegs pieces)
        int k = 0, hi = nseg - 1;
        while (k < hi) {
          const int mid = (k + hi) >> 1;
          if (kk < s_seg_end[mid]) hi = mid; else k = mid + 1;
        }
        const ExpressSeg& sg = s_seg[k].g;
        const int64_t j = kk - (k ? s_seg_end[k - 1] : 0);
        m_raw = sg.src ? sg.src[s * sg.stride + j] : (int32_t)(sg.start + j);
        m_bias = sg.logw * sqrt_d;
        m_vis = m_vis_nk = vis(s_seg[k].vlo, s_seg[k].vhi);
        m_piece = true;
      } else {
        m_cpos = (int32_t)(tile.causal_lo + (kk - F));
        m_kept = kept[m_cpos];
        // the tile's points whose C_0 starts at or before the candidate: a prefix
        int lo = 0, hi = (int)(q1 - q0);
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (s_c0[mid] <= m_cpos) lo = mid + 1; else hi = mid;
        }
        m_vis = vis(m_cpos, max((int64_t)m_cpos + 1, q0 + lo)) | 0x80000000u;
        m_vis_nk = vis(m_cpos, (int64_t)m_cpos + 1) | 0x80000000u;
      }
    }
  };
  gather_meta(0);
  for (int64_t ck = 0; ck < M; ck += KC) {
    const int kc = (int)min((int64_t)KC, M - ck);
    __syncthreads();
    if (threadIdx.x < KC) {
      int64_t r = m_piece ? (int64_t)m_raw : (m_cpos >= 0 ? (int64_t)m_cpos : 0);
      r = r < 0 ? 0 : (r >= n ? n - 1 : r);
      s_vis[threadIdx.x] = m_kept ? m_vis : m_vis_nk;
      s_row[threadIdx.x] = (int32_t)r;
      sB[threadIdx.x] = m_bias;
    }
    __syncthreads();
    for (int w = threadIdx.x; w < KC * WPR; w += 64 * PF_WAVES) {
      const int key = w / WPR, wi = w % WPR;
      uint4 kw = make_uint4(0, 0, 0, 0), vw = make_uint4(0, 0, 0, 0);
      if (key < kc) {
        const int64_t r = s_row[key];
        kw = reinterpret_cast<const uint4*>(Ks + r * D)[wi];
        if (!BF) vw = reinterpret_cast<const uint4*>(Vs + r * D)[wi];
      }
      *reinterpret_cast<uint4*>(sK + key * L::k_stride + wi * 16) = kw;
      if (!BF) *reinterpret_cast<uint4*>(sV + key * L::v_stride + wi * 16) = vw;
    }
    if (BF) {
      // V^T: each thread transposes 8 keys x 8 columns in registers and
      // writes 8 16-byte rows (one per column)
      for (int b = threadIdx.x; b < (KC / 8) * WPR; b += 64 * PF_WAVES) {
        const int kb = b / WPR, db = b % WPR;
        uint32_t v8[8][4];
#pragma unroll
        for (int r8 = 0; r8 < 8; ++r8) {
          const int key = kb * 8 + r8;
          uint4 x = make_uint4(0, 0, 0, 0);
          if (key < kc) x = reinterpret_cast<const uint4*>(Vs + (int64_t)s_row[key] * D)[db];
          v8[r8][0] = x.x; v8[r8][1] = x.y; v8[r8][2] = x.z; v8[r8][3] = x.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int k = e >> 1;
          uint4 o;
          if ((e & 1) == 0) {
            o.x = pack_lo(v8[0][k], v8[1][k]); o.y = pack_lo(v8[2][k], v8[3][k]);
            o.z = pack_lo(v8[4][k], v8[5][k]); o.w = pack_lo(v8[6][k], v8[7][k]);
          } else {
            o.x = pack_hi(v8[0][k], v8[1][k]); o.y = pack_hi(v8[2][k], v8[3][k]);
            o.z = pack_hi(v8[4][k], v8[5][k]); o.w = pack_hi(v8[6][k], v8[7][k]);
          }
          *reinterpret_cast<uint4*>(sV + (db * 8 + e) * L::v_stride + kb * 16) = o;
        }
      }
    }
    __syncthreads();
    if (ck + KC < M) gather_meta(ck + KC);

#pragma unroll
    for (int qt = 0; qt < PF_QT; ++qt) {
      const int64_t p = qw + qt * 16 + m16;  // this lane's point
      const uint32_t pl = (uint32_t)(p - q0);  // its offset in the tile
      const int li = (int)min(p - q0, (int64_t)QPB - 1);
      const float pw0 = p < q1 ? s_w0[li] * sqrt_d : 0.f;
      // the lane's 16 keys: bias where the point sees the key, else -inf
      float sc[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const uint4 w4 = *reinterpret_cast<const uint4*>(&s_vis[kt * 16 + 4 * g]);
        const float4 b4 = *reinterpret_cast<const float4*>(&sB[kt * 16 + 4 * g]);
        const uint32_t wv[4] = {w4.x, w4.y, w4.z, w4.w};
        const float kb[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool seen = pl >= (wv[i] & 0xffffu) && pl < ((wv[i] >> 16) & 0x7fffu);
          sc[kt][i] = seen ? ((int32_t)wv[i] < 0 ? pw0 : kb[i]) : -INFINITY;
        }
      }
      // (keeps the masks' LDS reads from being scheduled among the MFMAs
      // below, where their registers would push values out to scratch)
      __builtin_amdgcn_sched_barrier(0);
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        // the key tile's fragments from LDS for each query tile (re-read
        // rather than held: the registers keep two workgroups per CU)
        uint4 ak[NV];
        const uint4* pk = reinterpret_cast<const uint4*>(sK + (kt * 16 + m16) * L::k_stride);
#pragma unroll
        for (int v = 0; v < NV; ++v) ak[v] = pk[4 * v + g];
        floatx4_t z = {0.f, 0.f, 0.f, 0.f};
        z = mma_rows<T, D>(ak, Bq[qt], z);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sc[kt][i] += z[i];  // -inf stays -inf
          mx = fmaxf(mx, sc[kt][i]);
        }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(mrun[qt], mx);
      const float scale = (mrun[qt] == -INFINITY || mnew == -INFINITY)
                              ? 0.0f : __builtin_amdgcn_exp2f((mrun[qt] - mnew) * c2);
      mrun[qt] = mnew;
      // exp2(-inf) = 0 for the keys the point does not see; a row that sees
      // none yet subtracts 0 instead of -inf
      const float mref = mnew == -INFINITY ? 0.0f : mnew;
      float psum = 0.0f;
      float pr[4][4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = __builtin_amdgcn_exp2f((sc[kt][i] - mref) * c2);
          pr[kt][i] = pv;
          psum += pv;
        }
      lrun[qt] = lrun[qt] * scale + psum;
      // (the running maxima of most chunks stay put: no rescale then)
      if (__any(scale != 1.0f)) {
#pragma unroll
        for (int dt = 0; dt < D / 16; ++dt) acc[qt][dt] *= scale;
      }
      if (BF) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          float pv[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) pv[j] = pr[2 * c + (j >> 2)][j & 3];
          bf16x8_t bhi, blo;
          split_bf16x8(pv, bhi, blo);
#pragma unroll
          for (int dt = 0; dt < D / 16; ++dt) {
            const unsigned char* row = sV + (dt * 16 + m16) * L::v_stride;
            uint2 lo = *reinterpret_cast<const uint2*>(row + (32 * c + 4 * g) * 2);
            uint2 hi = *reinterpret_cast<const uint2*>(row + (32 * c + 16 + 4 * g) * 2);
            const bf16x8_t av = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bhi, acc[qt][dt], 0, 0, 0);
            acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, blo, acc[qt][dt], 0, 0, 0);
          }
        }
      } else {
#pragma unroll
        for (int kt = 0; kt < 4; ++kt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int key = kt * 16 + 4 * g + i;
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) {
              const float av = *reinterpret_cast<const float*>(sV + key * L::v_stride + (dt * 16 + m16) * 4);
              acc[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, pr[kt][i], acc[qt][dt], 0, 0, 0);
            }
          }
      }
    }
  }

#pragma unroll
  for (int qt = 0; qt < PF_QT; ++qt) {
    float l = lrun[qt];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const float inv = 1.0f / l;
    const int64_t q = qw + qt * 16 + m16;
    if (q < q1) {
      TO* orow = O + (s * n + q) * D;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt)
        store4<TO>(orow + dt * 16 + 4 * g, acc[qt][dt][0] * inv, acc[qt][dt][1] * inv,
                   acc[qt][dt][2] * inv, acc[qt][dt][3] * inv);
    }
  }
}

template <typename T, int D, typename TO>
hipError_t launch_prefill_t(const void* Q, const void* K, const void* V, int64_t S, int64_t n,
                            const PrefillTile* tiles, int64_t ntiles, const PrefillSeg* segs,
                            const int32_t* c0, const float* w0, const uint8_t* kept, void* O,
                            hipStream_t st) {
  dim3 grid((unsigned)ntiles, (unsigned)S), block(64 * PF_WAVES);
  hipLaunchKernelGGL((prefill_attn_kernel<T, D, TO>), grid, block, 0, st, (const T*)Q,
                     (const T*)K, (const T*)V, n, tiles, segs, c0, w0, kept, (TO*)O);
  return hipGetLastError();
}

template <typename T, typename TO>
hipError_t launch_prefill_d(int64_t d, const void* Q, const void* K, const void* V, int64_t S,
                            int64_t n, const PrefillTile* tiles, int64_t ntiles,
                            const PrefillSeg* segs, const int32_t* c0, const float* w0,
                            const uint8_t* kept, void* O, hipStream_t st) {
  switch (d) {
    case 32: return launch_prefill_t<T, 32, TO>(Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st);
    case 64: return launch_prefill_t<T, 64, TO>(Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st);
    case 128: return launch_prefill_t<T, 128, TO>(Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int D, typename TO>
hipError_t launch_attn_t(const void* Q, const void* K, const void* V, const int32_t* idx,
                         const float* logw, int64_t S, int64_t n, int64_t n_q, int64_t n_out,
                         void* O, hipStream_t st) {
  dim3 grid((unsigned)((n_q + QPB - 1) / QPB), (unsigned)S), block(64 * WAVES);
  if (logw)
    hipLaunchKernelGGL((coreset_attn_kernel<T, D, TO, true>), grid, block, 0, st, (const T*)Q,
                       (const T*)K, (const T*)V, idx, logw, n, n_q, (int)n_out, (TO*)O);
  else
    hipLaunchKernelGGL((coreset_attn_kernel<T, D, TO, false>), grid, block, 0, st, (const T*)Q,
                       (const T*)K, (const T*)V, idx, logw, n, n_q, (int)n_out, (TO*)O);
  return hipGetLastError();
}

template <typename T, typename TO>
hipError_t launch_attn_d(int64_t d, const void* Q, const void* K, const void* V,
                         const int32_t* idx, const float* logw, int64_t S, int64_t n,
                         int64_t n_q, int64_t n_out, void* O, hipStream_t st) {
  switch (d) {
    case 32: return launch_attn_t<T, 32, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
    case 64: return launch_attn_t<T, 64, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
    case 128: return launch_attn_t<T, 128, TO>(Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_prefill_attention(int dtype, int64_t d, int out_dtype, const void* Q,
                                    const void* K, const void* V, int64_t S, int64_t n,
                                    const PrefillTile* tiles, int64_t ntiles,
                                    const PrefillSeg* segs, const int32_t* c0, const float* w0,
                                    const uint8_t* kept, void* O, hipStream_t st) {
  if (ntiles < 1) return hipSuccess;
  if (dtype == 0)
    return out_dtype == 0
               ? launch_prefill_d<float, float>(d, Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st)
               : launch_prefill_d<float, bf16_t>(d, Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st);
  return out_dtype == 0
             ? launch_prefill_d<bf16_t, float>(d, Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st)
             : launch_prefill_d<bf16_t, bf16_t>(d, Q, K, V, S, n, tiles, ntiles, segs, c0, w0, kept, O, st);
}

hipError_t launch_attention(int dtype, int64_t d, int out_dtype, const void* Q, const void* K,
                            const void* V, const int32_t* idx, const float* logw, int64_t S,
                            int64_t n, int64_t n_q, int64_t n_out, void* O, hipStream_t st) {
  if (dtype == 0) {
    if (out_dtype == 0)
      return launch_attn_d<float, float>(d, Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
    return launch_attn_d<float, bf16_t>(d, Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  }
  bool used = false;
  hipError_t e = hipSuccess;
  if (d == 64)
    e = out_dtype == 0
            ? launch_attn_res_d<64, float>(n_out, Q, K, V, idx, logw, S, n, n_q, O, st, &used)
            : launch_attn_res_d<64, bf16_t>(n_out, Q, K, V, idx, logw, S, n, n_q, O, st, &used);
  else if (d == 128)
    e = out_dtype == 0
            ? launch_attn_res_d<128, float>(n_out, Q, K, V, idx, logw, S, n, n_q, O, st, &used)
            : launch_attn_res_d<128, bf16_t>(n_out, Q, K, V, idx, logw, S, n, n_q, O, st, &used);
  if (used) return e;
  if (out_dtype == 0)
    return launch_attn_d<bf16_t, float>(d, Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
  return launch_attn_d<bf16_t, bf16_t>(d, Q, K, V, idx, logw, S, n, n_q, n_out, O, st);
}

}  // namespace thin
