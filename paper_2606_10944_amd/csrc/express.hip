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

// dst[s * dst_stride + j] = start + j  (j < len)
__global__ void rows_iota_kernel(int32_t* dst, int64_t dst_stride, int64_t start, int64_t len) {
  const int64_t s = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < len) dst[s * dst_stride + j] = (int32_t)(start + j);
}

// dst[s * dst_stride + j] = src[s * src_stride + j]  (j < len)
__global__ void rows_copy_kernel(const int32_t* src, int64_t src_stride, int32_t* dst,
                                 int64_t dst_stride, int64_t len) {
  const int64_t s = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < len) dst[s * dst_stride + j] = src[s * src_stride + j];
}

// v_max of one Halve call (eq. katt over the rows it thins): the largest
// |V[s, idx[s, j], c]| over its N rows, as the float's bit pattern.  One
// workgroup per slice; a row is d * bytes / 16 16-byte words.
template <typename T>
__global__ __launch_bounds__(256) void vmax_rows_kernel(const T* V, int64_t ld, int64_t d,
                                                        const int32_t* idx, int64_t N,
                                                        uint32_t* vmax_bits) {
  const int64_t s = blockIdx.x;
  const int64_t wpr = d * Elem<T>::bytes / 16;
  const u32x4* base = reinterpret_cast<const u32x4*>(V + s * ld * d);
  uint32_t m = 0u;
  for (int64_t w = threadIdx.x; w < N * wpr; w += blockDim.x) {
    const int64_t row = idx[s * N + w / wpr];
    const u32x4 x = base[row * wpr + w % wpr];
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
  const float mf = wave_max(__uint_as_float(m));
  __shared__ float part[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) part[wave] = mf;
  __syncthreads();
  if (threadIdx.x == 0)
    vmax_bits[s] = __float_as_uint(fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3])));
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

}  // namespace

hipError_t launch_rows_iota(int32_t* dst, int64_t dst_stride, int64_t start, int64_t len,
                            int64_t S, hipStream_t st) {
  if (len <= 0) return hipSuccess;
  dim3 grid((unsigned)((len + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(rows_iota_kernel, grid, dim3(256), 0, st, dst, dst_stride, start, len);
  return hipGetLastError();
}

hipError_t launch_rows_copy(const int32_t* src, int64_t src_stride, int32_t* dst,
                            int64_t dst_stride, int64_t len, int64_t S, hipStream_t st) {
  if (len <= 0) return hipSuccess;
  dim3 grid((unsigned)((len + 255) / 256), (unsigned)S);
  hipLaunchKernelGGL(rows_copy_kernel, grid, dim3(256), 0, st, src, src_stride, dst, dst_stride,
                     len);
  return hipGetLastError();
}

hipError_t launch_vmax_rows(int dtype, const void* V, int64_t ld, int64_t d, const int32_t* idx,
                            int64_t N, int64_t S, uint32_t* vmax_bits, hipStream_t st) {
  if (dtype == 0)
    hipLaunchKernelGGL(vmax_rows_kernel<float>, dim3((unsigned)S), dim3(256), 0, st,
                       (const float*)V, ld, d, idx, N, vmax_bits);
  else
    hipLaunchKernelGGL(vmax_rows_kernel<bf16_t>, dim3((unsigned)S), dim3(256), 0, st,
                       (const bf16_t*)V, ld, d, idx, N, vmax_bits);
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
