// Device helpers of the Express cache (Sec. 3, Alg. 1 and 2): index-list
// moves, the per-call v_max of a Halve call and the layout of the weighted
// key list a point attends over (Alg. 5).  The Halve calls themselves are
// the KH rounds of compress.hip, one bucket per slice.
#include "common.hpp"
#include "launch.hpp"

namespace thin {

namespace {

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// dst[s * dst_stride + j] = src[s * src_stride + j]  (j < len)
__global__ void rows_copy_kernel(const int32_t* src, int64_t src_stride, int32_t* dst,
                                 int64_t dst_stride, int64_t len) {
  const int64_t s = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < len) dst[s * dst_stride + j] = src[s * src_stride + j];
}

// v_max of a Halve call (eq. katt over the rows it thins): the largest
// |V[s, row, c]| over its N rows idx[s * in_stride + t * N + j], as the
// float's bit pattern at vmax_bits[s * G + t].  One workgroup per call (G
// calls per slice); a row is d * bytes / 16 16-byte words.
template <typename T, int kU>
__global__ __launch_bounds__(256) void vmax_rows_kernel(const T* V, int64_t ld, int64_t d,
                                                        const int32_t* idx, int64_t in_stride,
                                                        int64_t N, int64_t G,
                                                        uint32_t* vmax_bits) {
  const int64_t s = blockIdx.x / G, t = blockIdx.x % G;
  const int64_t wpr = d * Elem<T>::bytes / 16;
  const u32x4* base = reinterpret_cast<const u32x4*>(V + s * ld * d);
  const int32_t* rows = idx + s * in_stride + t * N;
  uint32_t m = 0u;
  // kU words per thread per pass: every row index of a pass is requested,
  // then every word, so a pass waits for two memory latencies, not 2 kU
  // (wpr is a power of two for every supported d and element size)
  const int sh = __builtin_ctzll((unsigned long long)wpr);
  const int32_t total = (int32_t)(N * wpr);
  for (int32_t w0 = threadIdx.x; w0 < total; w0 += kU * (int32_t)blockDim.x) {
    int64_t row[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int32_t w = w0 + u * (int32_t)blockDim.x;
      row[u] = w < total ? (int64_t)rows[w >> sh] : -1;
    }
    u32x4 x[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int32_t w = w0 + u * (int32_t)blockDim.x;
      x[u] = row[u] >= 0 ? base[row[u] * wpr + (w & (int32_t)(wpr - 1))] : (u32x4){0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (Elem<T>::bytes == 4) {
          m = max(m, x[u][c] & 0x7fffffffu);
        } else {
          m = max(m, (x[u][c] << 16) & 0x7fffffffu);
          m = max(m, x[u][c] & 0x7fff0000u);
        }
      }
  }
  const float mf = wave_max(__uint_as_float(m));
  __shared__ float part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = mf;
  __syncthreads();
  if (threadIdx.x == 0)
    vmax_bits[blockIdx.x] = __float_as_uint(fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3])));
}

// The largest |V[s, r, c]| of every row r < n of every slice (rows n apart),
// as the float's bit pattern at absmax[s * n + r]: one thread per 16-byte
// word, the 2^wsh words of a row reduced by lane shuffles.  A Halve call's
// v_max is then the largest entry of its rows (vmax_table_kernel): the same
// integer maxima as vmax_rows_kernel, taken in another order.
template <typename T>
__global__ __launch_bounds__(256) void row_absmax_kernel(const T* V, int64_t words, int wsh,
                                                         uint32_t* absmax) {
  const int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t m = 0u;
  if (w < words) {
    const u32x4 x = reinterpret_cast<const u32x4*>(V)[w];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (Elem<T>::bytes == 4) {
        m = max(m, x[c] & 0x7fffffffu);
      } else {
        m = max(m, (x[c] << 16) & 0x7fffffffu);
        m = max(m, x[c] & 0x7fff0000u);
      }
    }
  }
  for (int off = 1; off < (1 << wsh); off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
  if (w < words && (w & ((1 << wsh) - 1)) == 0) absmax[w >> wsh] = m;
}

// v_max of G Halve calls per slice from the row table above: call t of slice
// s over the rows idx[s * in_stride + t * N + j] (negative: no row), into
// vmax_bits[s * G + t].  One workgroup per call.
__global__ __launch_bounds__(256) void vmax_table_kernel(const uint32_t* absmax, int64_t n,
                                                         const int32_t* idx, int64_t in_stride,
                                                         int64_t N, int64_t G,
                                                         uint32_t* vmax_bits) {
  const int64_t s = blockIdx.x / G, t = blockIdx.x % G;
  const uint32_t* tab = absmax + s * n;
  const int32_t* rows = idx + s * in_stride + t * N;
  uint32_t m = 0u;
  for (int64_t j = threadIdx.x; j < N; j += blockDim.x) {
    const int32_t r = rows[j];
    m = max(m, r >= 0 ? tab[r] : 0u);
  }
  const float mf = wave_max(__uint_as_float(m));
  __shared__ float part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = mf;
  __syncthreads();
  if (threadIdx.x == 0)
    vmax_bits[blockIdx.x] = __float_as_uint(fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3])));
}

// vmax_table_kernel for calls of at most 64 rows: one wave per call (call
// c = 4 blockIdx.x + wave, c < calls), lane j reads row j.
__global__ __launch_bounds__(256) void vmax_table_small_kernel(const uint32_t* absmax, int64_t n,
                                                               const int32_t* idx,
                                                               int64_t in_stride, int64_t N,
                                                               int64_t G, int64_t calls,
                                                               uint32_t* vmax_bits) {
  const int lane = threadIdx.x & 63;
  const int64_t c = 4 * (int64_t)blockIdx.x + (threadIdx.x >> 6);
  if (c >= calls) return;  // whole waves
  const int64_t s = c / G, t = c % G;
  uint32_t m = 0u;
  if (lane < N) {
    const int32_t r = idx[s * in_stride + t * N + lane];
    m = r >= 0 ? absmax[s * n + r] : 0u;
  }
  const float mf = wave_max(__uint_as_float(m));
  if (lane == 0) vmax_bits[c] = __float_as_uint(mf);
}

// Key j of slice s: the segment k with off_k <= j < off_k + len_k gives
// src_k[s * stride_k + j - off_k] (src_k null: start_k + j - off_k) and logw_k;
// slice s's keys start at s * out_stride.
__global__ void express_keys_kernel(ExpressSegs segs, int64_t m, int64_t out_stride, int32_t* idx,
                                    float* logw) {
  const int64_t s = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= m) return;
  int k = 0;
  int64_t off = 0;
  while (k + 1 < segs.n && j >= off + segs.seg[k].len) off += segs.seg[k++].len;
  const ExpressSeg& g = segs.seg[k];
  const int64_t r = j - off;
  idx[s * out_stride + j] = g.src ? g.src[s * g.stride + r] : (int32_t)(g.start + r);
  logw[s * out_stride + j] = g.logw;
}

// ---------------------------------------------------------------------------
// Weighted attention of one query per slice (a decoding step, Alg. 5) over
// the m keys of the cache segments (read in place: no key list is written),
// each key with its segment's log-weight.  The keys of a slice are split
// over `split` workgroups of 16 waves; a wave takes a contiguous run of keys
// and reads them with 16-byte loads, a key row spread over LPK lanes, so one
// load instruction brings 64 / LPK keys (4 bf16 rows of d = 128) and a wave
// keeps kDecUnroll such loads of K and of V in flight.  Each lane group of a
// key keeps an online softmax (log2 domain) of its keys; the groups merge by
// lane shuffles, the waves in LDS.  split == 1: the workgroup normalises and
// writes the output row itself (one launch per step); else it writes its
// unnormalised partial (max, sum, acc[D]) and a second kernel merges them.
// ---------------------------------------------------------------------------
#ifndef DEC_WAVES
#define DEC_WAVES 16
#endif
constexpr int kDecWaves = DEC_WAVES;
constexpr int kDecUnroll = 8;

// Row and log-weight of key j of slice s (segments as in express_keys_kernel).
// (k, off) is a cursor: segment k starts at key off; a lane's keys increase,
// so the cursor only moves forward.
__device__ __forceinline__ int64_t seg_key(const ExpressSegs& segs, int64_t s, int64_t j, int& k,
                                           int64_t& off, float* lw) {
  while (k + 1 < segs.n && j >= off + segs.seg[k].len) off += segs.seg[k++].len;
  const ExpressSeg& g = segs.seg[k];
  *lw = g.logw;
  return g.src ? (int64_t)g.src[s * g.stride + (j - off)] : g.start + (j - off);
}

// seg_key over a segment table staged in LDS.
__device__ __forceinline__ int64_t seg_key_lds(const ExpressSeg* seg, int n, int64_t s, int64_t j,
                                               int& k, int64_t& off, float* lw) {
  while (k + 1 < n && j >= off + seg[k].len) off += seg[k++].len;
  const ExpressSeg& g = seg[k];
  *lw = g.logw;
  return g.src ? (int64_t)g.src[s * g.stride + (j - off)] : g.start + (j - off);
}

// The EPW elements of a 16-byte word as floats.
template <typename T>
__device__ __forceinline__ void word_to_floats(const u32x4& w, float* out);
template <>
__device__ __forceinline__ void word_to_floats<float>(const u32x4& w, float* out) {
#pragma unroll
  for (int c = 0; c < 4; ++c) out[c] = __uint_as_float(w[c]);
}
template <>
__device__ __forceinline__ void word_to_floats<bf16_t>(const u32x4& w, float* out) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    out[2 * c] = __uint_as_float(w[c] << 16);
    out[2 * c + 1] = __uint_as_float(w[c] & 0xffff0000u);
  }
}

template <typename TO>
__device__ __forceinline__ void store_out(TO* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<bf16_t>(bf16_t* p, float v) {
  *reinterpret_cast<__bf16*>(p) = (__bf16)v;
}

// Merge of two online-softmax states (m, l, acc) in the log2 domain; an empty
// state has m = -inf.
template <int EPW>
__device__ __forceinline__ void softmax_merge(float& m, float& l, float* acc, float m2, float l2,
                                              const float* acc2) {
  const float M = fmaxf(m, m2);
  const float a = m == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m - M);
  const float b = m2 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m2 - M);
  l = l * a + l2 * b;
#pragma unroll
  for (int e = 0; e < EPW; ++e) acc[e] = acc[e] * a + acc2[e] * b;
  m = M;
}

template <typename T, int D, typename TO>
__global__ __launch_bounds__(64 * kDecWaves) void decode_attn_kernel(
    const T* __restrict__ Q, const T* __restrict__ K, const T* __restrict__ V, ExpressSegs segs,
    int64_t ld, int64_t m, int split, float* __restrict__ part, TO* __restrict__ O, int32_t* app,
    int64_t app_stride, int32_t app_val) {
  constexpr int LPK = D * Elem<T>::bytes / 16;  // lanes per key row (16 bytes each)
  constexpr int KPI = 64 / LPK;                 // keys per load instruction
  constexpr int EPW = 16 / Elem<T>::bytes;      // elements per 16-byte word
  static_assert(LPK >= 1 && LPK <= 64 && 64 % LPK == 0, "row of 16..1024 bytes");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int sub = lane / LPK, pos = lane % LPK;
  const int64_t s = blockIdx.y;
  const int64_t k0 = m * blockIdx.x / split, k1 = m * (blockIdx.x + 1) / split;
  // this wave's contiguous run of keys
  const int64_t per = (k1 - k0 + kDecWaves - 1) / kDecWaves;
  const int64_t w0 = min(k1, k0 + per * wave), w1 = min(k1, w0 + per);
  const float c2 = (float)(1.4426950408889634 / sqrt((double)D));
  const float l2e = 1.4426950408889634f;
  float q[EPW];
  word_to_floats<T>(reinterpret_cast<const u32x4*>(Q + s * D)[pos], q);
  const u32x4* Ks = reinterpret_cast<const u32x4*>(K + s * ld * D);
  const u32x4* Vs = reinterpret_cast<const u32x4*>(V + s * ld * D);
  // the segment table in LDS (the kernel argument is read through memory:
  // scanning it there would put a memory latency on every segment step)
  __shared__ ExpressSeg s_seg[kExpressMaxSegs];
  __shared__ int s_nseg;
  if (threadIdx.x < segs.n) s_seg[threadIdx.x] = segs.seg[threadIdx.x];
  if (threadIdx.x == 0) s_nseg = segs.n;
  __syncthreads();
  float mrun = -INFINITY, lrun = 0.f, acc[EPW];
#pragma unroll
  for (int e = 0; e < EPW; ++e) acc[e] = 0.f;
  int kseg = 0;
  int64_t koff = 0;
  for (int64_t j0 = w0; j0 < w1; j0 += KPI * kDecUnroll) {
    u32x4 kw[kDecUnroll], vw[kDecUnroll];
    float sc[kDecUnroll];
    int64_t r[kDecUnroll];
    // every row index of the batch first (the list reads are independent),
    // then every row: two dependent memory latencies per batch, not two per key
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const int64_t j = j0 + u * KPI + sub;
      const bool ok = j < w1;
      float lw = 0.f;
      r[u] = ok ? seg_key_lds(s_seg, s_nseg, s, j, kseg, koff, &lw) : -1;
      sc[u] = ok ? lw * l2e : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const bool ok = r[u] >= 0;
      kw[u] = ok ? Ks[r[u] * LPK + pos] : (u32x4){0u, 0u, 0u, 0u};
      vw[u] = ok ? Vs[r[u] * LPK + pos] : (u32x4){0u, 0u, 0u, 0u};
    }
    float mx = mrun;
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      float kf[EPW];
      word_to_floats<T>(kw[u], kf);
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < EPW; ++e) d = __builtin_fmaf(q[e], kf[e], d);
#pragma unroll
      for (int off = LPK / 2; off >= 1; off >>= 1) d += __shfl_xor(d, off);
      sc[u] = sc[u] == -INFINITY ? -INFINITY : __builtin_fmaf(d, c2, sc[u]);
      mx = fmaxf(mx, sc[u]);
    }
    if (mx == -INFINITY) continue;  // nothing of positive weight yet
    const float scale = mrun == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mrun - mx);
    lrun *= scale;
#pragma unroll
    for (int e = 0; e < EPW; ++e) acc[e] *= scale;
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const float p = sc[u] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sc[u] - mx);
      float vf[EPW];
      word_to_floats<T>(vw[u], vf);
      lrun += p;
#pragma unroll
      for (int e = 0; e < EPW; ++e) acc[e] = __builtin_fmaf(p, vf[e], acc[e]);
    }
    mrun = mx;
  }
  // the wave's KPI key groups merge into lanes 0..LPK-1
#pragma unroll
  for (int off = LPK; off < 64; off <<= 1) {
    const float m2 = __shfl_xor(mrun, off), l2 = __shfl_xor(lrun, off);
    float a2[EPW];
#pragma unroll
    for (int e = 0; e < EPW; ++e) a2[e] = __shfl_xor(acc[e], off);
    softmax_merge<EPW>(mrun, lrun, acc, m2, l2, a2);
  }
  __shared__ float s_m[kDecWaves], s_l[kDecWaves], s_acc[kDecWaves][D];
  if (lane == 0) {
    s_m[wave] = mrun;
    s_l[wave] = lrun;
  }
  if (lane < LPK) {
#pragma unroll
    for (int e = 0; e < EPW; ++e) s_acc[wave][pos * EPW + e] = acc[e];
  }
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, s_m[w]);
  const int c = threadIdx.x;
  if (c < D) {
    float a = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      const float f = s_m[w] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s_m[w] - M);
      a = __builtin_fmaf(s_acc[w][c], f, a);
      L = __builtin_fmaf(s_l[w], f, L);
    }
    if (split == 1) {
      store_out<TO>(O + s * D + c, a / L);
    } else {
      float* out = part + (s * split + blockIdx.x) * (int64_t)(D + 2);
      out[2 + c] = a;
      if (c == 0) {
        out[0] = M;
        out[1] = L;
      }
    }
  }
  if (split == 1 && app && threadIdx.x == 0) app[s * app_stride] = app_val;
}

// One workgroup per slice: the partials' maxima and sums are staged in LDS
// (one load each), then thread c merges column c of every partial.  With
// app non-null, thread 0 also writes the point's position app_val to
// app[s * app_stride] (the point entering its cache list).
template <int D, typename TO>
__global__ __launch_bounds__(128) void decode_attn_merge_kernel(const float* __restrict__ part,
                                                                int split, TO* __restrict__ O,
                                                                int32_t* app, int64_t app_stride,
                                                                int32_t app_val) {
  const int64_t s = blockIdx.x;
  if (app && threadIdx.x == 0) app[s * app_stride] = app_val;
  const float* p = part + s * split * (int64_t)(D + 2);
  __shared__ float s_w[kDecodeMaxSplit], s_l[kDecodeMaxSplit];
  __shared__ float s_M;
  if (threadIdx.x < split) {
    s_w[threadIdx.x] = p[threadIdx.x * (D + 2)];
    s_l[threadIdx.x] = p[threadIdx.x * (D + 2) + 1];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = -INFINITY;
    for (int k = 0; k < split; ++k) M = fmaxf(M, s_w[k]);
    s_M = M;
  }
  __syncthreads();
  if (threadIdx.x < split)  // each partial's scale exp2(m_k - M), 0 for an empty one
    s_w[threadIdx.x] = s_w[threadIdx.x] == -INFINITY ? 0.f
                                                     : __builtin_amdgcn_exp2f(s_w[threadIdx.x] - s_M);
  __syncthreads();
  float L = 0.f;
  for (int k = 0; k < split; ++k) L = __builtin_fmaf(s_l[k], s_w[k], L);
  for (int c = threadIdx.x; c < D; c += blockDim.x) {
    float v[kDecodeMaxSplit];
#pragma unroll
    for (int k = 0; k < kDecodeMaxSplit; ++k) v[k] = k < split ? p[k * (D + 2) + 2 + c] : 0.f;
    float a = 0.f;
#pragma unroll
    for (int k = 0; k < kDecodeMaxSplit; ++k) a = __builtin_fmaf(v[k], k < split ? s_w[k] : 0.f, a);
    store_out<TO>(O + s * D + c, a / L);
  }
}

struct Append {
  int32_t* dst;
  int64_t stride;
  int32_t val;
};

template <typename T, int D, typename TO>
hipError_t launch_decode_t(const void* Q, const void* K, const void* V, const ExpressSegs& segs,
                           int64_t S, int64_t ld, int64_t m, int split, float* part, void* O,
                           const Append& ap, hipStream_t st) {
  hipLaunchKernelGGL((decode_attn_kernel<T, D, TO>), dim3((unsigned)split, (unsigned)S),
                     dim3(64 * kDecWaves), 0, st, (const T*)Q, (const T*)K, (const T*)V, segs, ld,
                     m, split, part, (TO*)O, ap.dst, ap.stride, ap.val);
  if (split > 1)
    hipLaunchKernelGGL((decode_attn_merge_kernel<D, TO>), dim3((unsigned)S), dim3(128), 0, st,
                       (const float*)part, split, (TO*)O, ap.dst, ap.stride, ap.val);
  return hipGetLastError();
}

template <typename T, typename TO>
hipError_t launch_decode_d(int64_t d, const void* Q, const void* K, const void* V,
                           const ExpressSegs& g, int64_t S, int64_t ld, int64_t m, int split,
                           float* part, void* O, const Append& ap, hipStream_t st) {
  switch (d) {
    case 32: return launch_decode_t<T, 32, TO>(Q, K, V, g, S, ld, m, split, part, O, ap, st);
    case 64: return launch_decode_t<T, 64, TO>(Q, K, V, g, S, ld, m, split, part, O, ap, st);
    case 128: return launch_decode_t<T, 128, TO>(Q, K, V, g, S, ld, m, split, part, O, ap, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_attention_split(int64_t m) {
  const int64_t sp = (m + kDecodeKeysPerGroup - 1) / kDecodeKeysPerGroup;
  return (int)(sp < 1 ? 1 : (sp > kDecodeMaxSplit ? kDecodeMaxSplit : sp));
}

hipError_t launch_decode_attention(int dtype, int64_t d, int out_dtype, const void* Q,
                                   const void* K, const void* V, const ExpressSegs& g, int64_t S,
                                   int64_t ld, int64_t m, float* part, void* O, int32_t* app,
                                   int64_t app_stride, int32_t app_val, hipStream_t st) {
  if (m < 1 || g.n < 1) return hipErrorInvalidValue;
  const int split = decode_attention_split(m);
  const Append ap{app, app_stride, app_val};
  if (dtype == 0)
    return out_dtype == 0
               ? launch_decode_d<float, float>(d, Q, K, V, g, S, ld, m, split, part, O, ap, st)
               : launch_decode_d<float, bf16_t>(d, Q, K, V, g, S, ld, m, split, part, O, ap, st);
  return out_dtype == 0
             ? launch_decode_d<bf16_t, float>(d, Q, K, V, g, S, ld, m, split, part, O, ap, st)
             : launch_decode_d<bf16_t, bf16_t>(d, Q, K, V, g, S, ld, m, split, part, O, ap, st);
}

hipError_t launch_rows_copy(const int32_t* src, int64_t src_stride, int32_t* dst,
                            int64_t dst_stride, int64_t len, int64_t S, hipStream_t st) {
  if (len <= 0) return hipSuccess;
  dim3 grid((unsigned)((len + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(rows_copy_kernel, grid, dim3(256), 0, st, src, src_stride, dst, dst_stride,
                     len);
  return hipGetLastError();
}

hipError_t launch_row_absmax(int dtype, const void* V, int64_t n, int64_t d, int64_t S,
                             uint32_t* absmax, hipStream_t st) {
  const int64_t wpr = d * (dtype == 0 ? 4 : 2) / 16;  // a power of two, 1..64
  if (wpr < 1 || wpr > 64 || (wpr & (wpr - 1)) != 0) return hipErrorInvalidValue;
  const int64_t words = S * n * wpr;
  if (words <= 0) return hipSuccess;
  const int64_t blocks = (words + 255) / 256;
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const int wsh = __builtin_ctzll((unsigned long long)wpr);
  if (dtype == 0)
    hipLaunchKernelGGL((row_absmax_kernel<float>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const float*)V, words, wsh, absmax);
  else
    hipLaunchKernelGGL((row_absmax_kernel<bf16_t>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const bf16_t*)V, words, wsh, absmax);
  return hipGetLastError();
}

hipError_t launch_vmax_table(const uint32_t* absmax, int64_t n, const int32_t* idx,
                             int64_t in_stride, int64_t N, int64_t G, int64_t S,
                             uint32_t* vmax_bits, hipStream_t st) {
  if (S * G <= 0) return hipSuccess;
  if (N <= 64) {  // calls of at most 64 rows: one wave each, four to a workgroup
    hipLaunchKernelGGL(vmax_table_small_kernel, dim3((unsigned)((S * G + 3) / 4)), dim3(256), 0, st,
                       absmax, n, idx, in_stride, N, G, S * G, vmax_bits);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(vmax_table_kernel, dim3((unsigned)(S * G)), dim3(256), 0, st, absmax, n, idx,
                     in_stride, N, G, vmax_bits);
  return hipGetLastError();
}

hipError_t launch_vmax_rows(int dtype, const void* V, int64_t ld, int64_t d, const int32_t* idx,
                            int64_t in_stride, int64_t N, int64_t G, int64_t S,
                            uint32_t* vmax_bits, hipStream_t st) {
  // a call's words are counted in 32 bits
  const int64_t words = N * d * (dtype == 0 ? 4 : 2) / 16;
  if (words >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(S * G));
  // calls of at most two words per thread take one word per pass
  if (dtype == 0) {
    if (words <= 512)
      hipLaunchKernelGGL((vmax_rows_kernel<float, 1>), grid, dim3(256), 0, st, (const float*)V, ld,
                         d, idx, in_stride, N, G, vmax_bits);
    else
      hipLaunchKernelGGL((vmax_rows_kernel<float, 8>), grid, dim3(256), 0, st, (const float*)V, ld,
                         d, idx, in_stride, N, G, vmax_bits);
  } else {
    if (words <= 512)
      hipLaunchKernelGGL((vmax_rows_kernel<bf16_t, 1>), grid, dim3(256), 0, st, (const bf16_t*)V,
                         ld, d, idx, in_stride, N, G, vmax_bits);
    else
      hipLaunchKernelGGL((vmax_rows_kernel<bf16_t, 8>), grid, dim3(256), 0, st, (const bf16_t*)V,
                         ld, d, idx, in_stride, N, G, vmax_bits);
  }
  return hipGetLastError();
}

hipError_t launch_express_keys(const ExpressSegs& segs, int64_t S, int64_t m, int64_t out_stride,
                               int32_t* idx, float* logw, hipStream_t st) {
  if (m <= 0 || segs.n < 1 || out_stride < m) return hipErrorInvalidValue;
  dim3 grid((unsigned)((m + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(express_keys_kernel, grid, dim3(256), 0, st, segs, m, out_stride, idx, logw);
  return hipGetLastError();
}

}  // namespace thin
