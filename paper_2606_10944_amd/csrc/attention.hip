// Coreset attention on gfx950: every query of a slice attends over the n_out
// rows idx[s, :] of that slice's K/V (Sec. 2.1 eq. unmaskedatt on the
// coreset; eq. def:att_approx with equal weights, which cancel).
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
constexpr double kLog2e = 1.44269504088896340736;

template <typename T, int D>
struct AttnLds {
  // K chunk, row-major, padded by 16 bytes per row.
  static constexpr int k_stride = D * Elem<T>::bytes + 16;
  // V chunk: bf16 is stored transposed [D][KC] (+8 elements pad), fp32 row-major.
  static constexpr int v_stride = Elem<T>::bytes == 2 ? (KC + 8) * 2 : D * 4 + 16;
  static constexpr int v_rows = Elem<T>::bytes == 2 ? D : KC;
  static constexpr int bytes = KC * k_stride + v_rows * v_stride;
};

template <typename TO>
__device__ __forceinline__ void store4(TO* p, float a, float b, float c, float d);

template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  uint2 w;
  w.x = (uint32_t)float_to_bf16(a) | ((uint32_t)float_to_bf16(b) << 16);
  w.y = (uint32_t)float_to_bf16(c) | ((uint32_t)float_to_bf16(d) << 16);
  *reinterpret_cast<uint2*>(p) = w;
}

template <typename T, int D, typename TO>
__global__ __launch_bounds__(64 * WAVES) void coreset_attn_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V,
    const int32_t* __restrict__ idx, int64_t n, int64_t n_q, int n_out, TO* __restrict__ O) {
  constexpr int NV = Frag<T, D>::NV;
  constexpr bool BF = Elem<T>::bytes == 2;
  using L = AttnLds<T, D>;
  __shared__ __align__(16) unsigned char lds[L::bytes];
  unsigned char* sK = lds;
  unsigned char* sV = lds + KC * L::k_stride;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m16 = lane & 15, g = lane >> 4;
  const int64_t s = blockIdx.y;
  const int64_t q0 = (int64_t)blockIdx.x * QPB + wave * 16 * QT;
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
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = kt * 16 + 4 * g + i;
          sc[kt][i] = key < kc ? z[i] : -INFINITY;
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
          uint16_t hb[8], lb[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float pv = pr[2 * c + (j >> 2)][j & 3];
            hb[j] = float_to_bf16(pv);
            lb[j] = float_to_bf16(pv - bf16_to_float(hb[j]));
          }
          uint4 hw, lw;
          hw.x = (uint32_t)hb[0] | ((uint32_t)hb[1] << 16);
          hw.y = (uint32_t)hb[2] | ((uint32_t)hb[3] << 16);
          hw.z = (uint32_t)hb[4] | ((uint32_t)hb[5] << 16);
          hw.w = (uint32_t)hb[6] | ((uint32_t)hb[7] << 16);
          lw.x = (uint32_t)lb[0] | ((uint32_t)lb[1] << 16);
          lw.y = (uint32_t)lb[2] | ((uint32_t)lb[3] << 16);
          lw.z = (uint32_t)lb[4] | ((uint32_t)lb[5] << 16);
          lw.w = (uint32_t)lb[6] | ((uint32_t)lb[7] << 16);
          const bf16x8_t bhi = __builtin_bit_cast(bf16x8_t, hw);
          const bf16x8_t blo = __builtin_bit_cast(bf16x8_t, lw);
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

template <typename T, int D, typename TO>
hipError_t launch_attn_t(const void* Q, const void* K, const void* V, const int32_t* idx,
                         int64_t S, int64_t n, int64_t n_q, int64_t n_out, void* O,
                         hipStream_t st) {
  dim3 grid((unsigned)((n_q + QPB - 1) / QPB), (unsigned)S), block(64 * WAVES);
  hipLaunchKernelGGL((coreset_attn_kernel<T, D, TO>), grid, block, 0, st, (const T*)Q,
                     (const T*)K, (const T*)V, idx, n, n_q, (int)n_out, (TO*)O);
  return hipGetLastError();
}

template <typename T, typename TO>
hipError_t launch_attn_d(int64_t d, const void* Q, const void* K, const void* V,
                         const int32_t* idx, int64_t S, int64_t n, int64_t n_q, int64_t n_out,
                         void* O, hipStream_t st) {
  switch (d) {
    case 32: return launch_attn_t<T, 32, TO>(Q, K, V, idx, S, n, n_q, n_out, O, st);
    case 64: return launch_attn_t<T, 64, TO>(Q, K, V, idx, S, n, n_q, n_out, O, st);
    case 128: return launch_attn_t<T, 128, TO>(Q, K, V, idx, S, n, n_q, n_out, O, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attention(int dtype, int64_t d, int out_dtype, const void* Q, const void* K,
                            const void* V, const int32_t* idx, int64_t S, int64_t n,
                            int64_t n_q, int64_t n_out, void* O, hipStream_t st) {
  if (dtype == 0) {
    if (out_dtype == 0) return launch_attn_d<float, float>(d, Q, K, V, idx, S, n, n_q, n_out, O, st);
    return launch_attn_d<float, bf16_t>(d, Q, K, V, idx, S, n, n_q, n_out, O, st);
  }
  if (out_dtype == 0) return launch_attn_d<bf16_t, float>(d, Q, K, V, idx, S, n, n_q, n_out, O, st);
  return launch_attn_d<bf16_t, bf16_t>(d, Q, K, V, idx, S, n, n_q, n_out, O, st);
}

}  // namespace thin
