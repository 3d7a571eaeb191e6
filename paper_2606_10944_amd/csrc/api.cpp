// C ABI of the thinning library: planning, argument validation and the
// level-synchronous launch sequence of the compress path.
#include <math.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <new>
#include <tuple>
#include <vector>
#include <stdint.h>
#include <string.h>

#include "../../include/thin.h"
#include "launch.hpp"

namespace {

constexpr int64_t kMaxBucket = 8192;  // the decision pass keeps a bucket's per-pair alpha in LDS
constexpr int64_t kMaxRows = (int64_t)1 << 30;
constexpr int64_t kMaxSlices = 65535;  // the per-slice kernels index slices by grid y

struct Levels {
  int64_t n = 0;
  int64_t n_kept = 0;
  int32_t L = 0;
  int32_t mc = 0;
  bool sub = false;
  int64_t U = 0;
  int64_t n_r[64];
  int64_t G[64];
  int64_t N[64];
  int64_t max_bucket = 0;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool supported_d(int64_t d) { return d == 32 || d == 64 || d == 128; }

// Integer planning of one compress call; false if no valid level structure.
bool make_levels(int64_t n, int64_t n_out, int32_t g, Levels* lv) {
  if (n < 1 || n > kMaxRows || n_out < 1 || n_out > n || g < 0) return false;
  int32_t L = 0;
  while ((n_out << (L + 1)) <= n) ++L;
  lv->L = L;
  lv->n = n;
  lv->n_kept = n_out << L;
  lv->sub = lv->n_kept < n;
  lv->mc = L - (g < L ? g : L);
  lv->U = (lv->sub ? lv->n_kept : 0) + (lv->n_kept - n_out);
  lv->max_bucket = 0;
  for (int32_t r = 0; r < L; ++r) {
    const int64_t n_r = lv->n_kept >> r;
    const int32_t e = L - g - 1 - r;
    const int64_t G = e > 0 ? ((int64_t)1 << (2 * e)) : 1;
    if (n_r % G != 0) return false;
    const int64_t N = n_r / G;
    if (N < 2 || (N & 1)) return false;
    lv->n_r[r] = n_r;
    lv->G[r] = G;
    lv->N[r] = N;
    if (N > lv->max_bucket) lv->max_bucket = N;
  }
  return true;
}

// Pair scores of one round live in a region of at most kScoreCap bytes (or
// one bucket's worth, if larger); rounds whose buckets need more run in
// several launches.
constexpr size_t kScoreCap = (size_t)2 << 30;

size_t score_bytes(int64_t N) { return thin::halve_score_bytes(N); }

size_t score_region(int64_t S, int64_t d, const Levels& lv, size_t cap_bytes = kScoreCap) {
  size_t region = 0;
  // rounds whose buckets run as one local launch (for either dtype) need none
  const int64_t local = std::min(thin::halve_local_rows(0, d), thin::halve_local_rows(1, d));
  for (int32_t r = 0; r < lv.L; ++r) {
    if (lv.N[r] <= local) continue;
    const size_t per = score_bytes(lv.N[r]);
    const size_t all = (size_t)(S * lv.G[r]) * per;
    const size_t cap = per > cap_bytes ? per : cap_bytes;
    const size_t need = all < cap ? all : cap;
    if (need > region) region = need;
  }
  return region;
}

// Per-block row-scale maxima of the largest round (floats).
size_t block_scales(int64_t S, const Levels& lv) {
  size_t m = 1;
  for (int32_t r = 0; r < lv.L; ++r)
    m = std::max(m, (size_t)(S * lv.G[r]) * (size_t)((lv.N[r] + 63) / 64));
  return m;
}

// Decision helpers' sizes over the rounds that may use them (thin::pass_helpers):
// tagged decision words, chunk flags, partial alphas.
struct HelperSizes {
  size_t masks = 0, flags = 0, alphas = 0;
};
HelperSizes helper_sizes(int64_t S, const Levels& lv) {
  HelperSizes h;
  for (int32_t r = 0; r < lv.L; ++r) {
    const int64_t buckets = S * lv.G[r], P = lv.N[r] / 2;
    if (buckets > thin::kHelperMaxBuckets || P < thin::kHelperMinPairs || P % 64 != 0) continue;
    h.masks = std::max(h.masks, (size_t)(buckets * ((P + 31) / 32)));
    h.flags = std::max(h.flags, (size_t)(buckets * ((P + 63) / 64)));
    h.alphas = std::max(h.alphas, (size_t)(buckets * P));
  }
  return h;
}

struct Workspace {
  int32_t* status;  // the device status word (thin.h), first in every workspace
  uint32_t* vmax_bits;
  uint64_t* gmask;  // decision helpers (null when no round may use them); zeroed with vmax_bits
  uint32_t* gflag;
  uint64_t* galpha;
  int64_t zero_words;  // words from vmax_bits through gflag
  int32_t* buf_a;  // [S, n_kept]
  int32_t* buf_b;  // [S, n_kept / 2]
  float* lbt;      // [S, n_kept / 2]
  float* h2;       // [S, n_kept / 2]
  float* rowh2;    // [S, n]
  float* mB;       // [buckets, ceil(N / 64)] of the largest round
  float* E;        // score region
  size_t e_bytes;
  size_t bytes;
};

Workspace carve(void* base, int64_t S, int64_t d, const Levels& lv, size_t cap = kScoreCap) {
  Workspace w;
  unsigned char* p = static_cast<unsigned char*>(base);
  const size_t pairs = (size_t)S * (size_t)(lv.n_kept / 2);
  size_t off = 0;
  w.status = reinterpret_cast<int32_t*>(p + off);
  off += 256;
  w.vmax_bits = reinterpret_cast<uint32_t*>(p + off);
  const size_t vmax_off = off;
  off += align256((size_t)S * 4);
  const HelperSizes hs = helper_sizes(S, lv);
  w.gmask = hs.masks ? reinterpret_cast<uint64_t*>(p + off) : nullptr;
  off += align256(hs.masks * 8);
  w.gflag = hs.flags ? reinterpret_cast<uint32_t*>(p + off) : nullptr;
  off += align256(hs.flags * 4);
  w.zero_words = (int64_t)((off - vmax_off) / 4);
  w.galpha = hs.alphas ? reinterpret_cast<uint64_t*>(p + off) : nullptr;
  off += align256(hs.alphas * 8);
  w.buf_a = reinterpret_cast<int32_t*>(p + off);
  off += align256((size_t)S * (size_t)lv.n_kept * 4);
  w.buf_b = reinterpret_cast<int32_t*>(p + off);
  off += align256(pairs * 4);
  w.lbt = reinterpret_cast<float*>(p + off);
  off += align256(pairs * 4);
  w.h2 = reinterpret_cast<float*>(p + off);
  off += align256(pairs * 4);
  w.rowh2 = reinterpret_cast<float*>(p + off);
  off += align256((size_t)S * (size_t)lv.n * 4);
  w.mB = reinterpret_cast<float*>(p + off);
  off += align256(block_scales(S, lv) * 4);
  w.E = reinterpret_cast<float*>(p + off);
  w.e_bytes = score_region(S, d, lv, cap);
  off += align256(w.e_bytes);
  w.bytes = off;
  return w;
}

size_t workspace_size(int64_t S, int64_t d, const Levels& lv, size_t cap = kScoreCap) {
  return carve(nullptr, S, d, lv, cap).bytes;
}

// The launch observer is a diagnostic of the calling thread (thread-local):
// calls from other threads never see it.
thread_local thin_launch_hook_t g_hook = nullptr;
thread_local void* g_hook_ctx = nullptr;

// Enqueue one launch between the observer's two calls.
template <typename F>
hipError_t observed(int32_t kernel, int32_t round, hipStream_t st, F&& launch) {
  if (g_hook) g_hook(g_hook_ctx, kernel, round, 0, st);
  const hipError_t e = launch();
  if (g_hook) g_hook(g_hook_ctx, kernel, round, 1, st);
  return e;
}

// One KH round over the S*G buckets described by `a`: one local launch for
// buckets up to the local kernel's size (however many: with 4096 buckets of
// 256 rows the local launch beats scores + decisions by ~5 %, with 16384 of
// 16 rows or 4096 of 64 rows by 2-2.5x), else pair scores then decisions, in
// as many launches as the score region (e_bytes) needs.
hipError_t kh_round(int32_t dtype, int64_t d, thin::HalveArgs a, int64_t buckets, size_t e_bytes,
                    int32_t r, hipStream_t st) {
  if (a.N <= thin::halve_local_rows(dtype, d)) {
    a.b0 = 0;
    return observed(THIN_KERNEL_LOCAL, r, st,
                    [&] { return thin::launch_local(dtype, d, a, buckets, st); });
  }
  const size_t per = thin::halve_score_bytes(a.N);
  int64_t chunk = (int64_t)(e_bytes / per);
  if (chunk < 1) chunk = 1;
  if (chunk < buckets) {  // several launches: the helpers' tags are per round
    a.gmask = nullptr;
    a.gflag = nullptr;
    a.galpha = nullptr;
  }
  hipError_t e = hipSuccess;
  for (int64_t b0 = 0; b0 < buckets && e == hipSuccess; b0 += chunk) {
    a.b0 = b0;
    const int64_t nbk = buckets - b0 < chunk ? buckets - b0 : chunk;
    e = observed(THIN_KERNEL_SCORES, r, st, [&] { return thin::launch_scores(dtype, d, a, nbk, st); });
    if (e == hipSuccess)
      e = observed(THIN_KERNEL_DECIDE, r, st, [&] { return thin::launch_decide(a, nbk, st); });
  }
  return e;
}

int check_shape(int64_t B, int64_t H, int64_t n, int64_t d) {
  if (B < 1 || H < 1 || n < 1 || n > kMaxRows) return THIN_EINVAL;
  if (B * H > kMaxSlices) return THIN_EINVAL;
  if (!supported_d(d)) return THIN_EINVAL;
  return THIN_OK;
}

int compress_impl(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H, int64_t n,
                  int64_t d, int64_t n_out, int32_t g, const float* uniforms, int64_t n_uniforms,
                  int32_t* idx_out, void* workspace, size_t workspace_bytes, uint8_t* trace,
                  int64_t trace_len, int32_t halve, const double* delta, int64_t n_sinks,
                  int64_t n_window, float* logw_out, void* stream, size_t cap = kScoreCap) {
  int rc = check_shape(B, H, n, d);
  if (rc) return rc;
  if (dtype != THIN_FP32 && dtype != THIN_BF16) return THIN_EDTYPE;
  if (n_sinks < 0 || n_window < 0 || n_sinks > n || n_window > n - n_sinks) return THIN_EINVAL;
  // the rows between the sinks and the window are thinned as a dataset of their own
  const int64_t nm = n - n_sinks - n_window;
  Levels lv;
  if (!make_levels(nm, n_out, g, &lv) || lv.max_bucket > kMaxBucket) return THIN_EINVAL;
  if (!K || !V || !idx_out) return THIN_EINVAL;
  const int64_t S = B * H;
  const int64_t Utot = S * lv.U;
  if (Utot > 0 && !uniforms) return THIN_EINVAL;
  if (n_uniforms < Utot) return THIN_EUNIFORMS;
  if (trace && trace_len < Utot) return THIN_EINVAL;
  if (halve != THIN_HALVE_KH && halve != THIN_HALVE_UNIFORM) return THIN_EINVAL;
  if (halve == THIN_HALVE_KH && delta)
    for (int32_t r = 0; r < lv.L; ++r)
      if (!(delta[r] > 0.0 && delta[r] <= 1.0)) return THIN_EINVAL;
  if (!workspace || workspace_bytes < workspace_size(S, d, lv, cap)) return THIN_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return THIN_EWORKSPACE;
  Workspace ws = carve(workspace, S, d, lv, cap);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t esz = dtype == THIN_FP32 ? 4 : 2;
  const void* Km = static_cast<const unsigned char*>(K) + (size_t)n_sinks * (size_t)d * esz;
  const void* Vm = static_cast<const unsigned char*>(V) + (size_t)n_sinks * (size_t)d * esz;
  // With exact rows the last round writes the coreset to whichever index
  // buffer it does not read, and one more launch lays out the output.
  const bool assemble = n_sinks > 0 || n_window > 0 || logw_out;
  auto last_out = [&](const int32_t* in) {
    return assemble ? (in == ws.buf_b ? ws.buf_a : ws.buf_b) : idx_out;
  };

  hipError_t e = hipSuccess;
  auto ok = [&](hipError_t x) {
    if (x != hipSuccess && e == hipSuccess) e = x;
    return e == hipSuccess;
  };
  if (trace)
    ok(observed(THIN_KERNEL_TRACE_CLEAR, -1, st, [&] { return thin::launch_zero_u8(trace, Utot, st); }));
  if (lv.sub)
    ok(observed(THIN_KERNEL_SUBSAMPLE, -1, st, [&] {
      return thin::launch_subsample(S, nm, lv.n_kept, uniforms, lv.U, ws.buf_a, st);
    }));
  const int32_t* cur = lv.sub ? ws.buf_a : nullptr;
  // the status word is cleared by the v_max launch of the KH path; calls
  // that make no KH decision clear it here
  if (lv.L == 0 || halve != THIN_HALVE_KH)
    ok(observed(THIN_KERNEL_STATUS, -1, st,
                [&] { return thin::launch_zero_status(ws.status, st); }));
  if (lv.L == 0) {
    if (!assemble)
      ok(observed(THIN_KERNEL_FILL, -1, st, [&] {
        return thin::launch_fill_rows(S, n_out, cur, lv.n_kept, idx_out, st);
      }));
  } else if (halve == THIN_HALVE_UNIFORM && thin::uniform_fused_ok(lv.n_kept)) {
    int32_t* out = last_out(cur);
    ok(observed(THIN_KERNEL_UNIFORM, -1, st, [&] {
      return thin::launch_uniform_compress(S, lv.n_kept, lv.L, cur, uniforms, lv.U,
                                           lv.sub ? lv.n_kept : 0, out, n_out, trace, st);
    }));
    cur = out;
  } else if (halve == THIN_HALVE_UNIFORM) {
    int64_t u_off = lv.sub ? lv.n_kept : 0;
    for (int32_t r = 0; r < lv.L && e == hipSuccess; ++r) {
      int32_t* out = (r == lv.L - 1) ? last_out(cur) : (cur == ws.buf_b ? ws.buf_a : ws.buf_b);
      ok(observed(THIN_KERNEL_UNIFORM, r, st, [&] {
        return thin::launch_uniform_halve(S, lv.n_r[r], cur, uniforms, lv.U, u_off, out, trace,
                                          st);
      }));
      u_off += lv.n_r[r] / 2;
      cur = out;
    }
  } else {
    ok(observed(THIN_KERNEL_VMAX, -1, st, [&] {
      return thin::launch_vmax(dtype, Vm, S, nm, n, d, ws.vmax_bits, st, ws.status, ws.zero_words);
    }));
    int64_t u_off = lv.sub ? lv.n_kept : 0;
    for (int32_t r = 0; r < lv.L && e == hipSuccess; ++r) {
      int32_t* out = (r == lv.L - 1) ? last_out(cur) : (cur == ws.buf_b ? ws.buf_a : ws.buf_b);
      thin::HalveArgs a{};
      a.K = Km;
      a.V = Vm;
      a.n = nm;
      a.ld = n;
      a.vmax_bits = ws.vmax_bits;
      a.idx_in = cur;
      a.n_r = lv.n_r[r];
      a.N = (int32_t)lv.N[r];
      a.G = (int32_t)lv.G[r];
      a.S = S;
      a.idx_out = out;
      a.U = uniforms;
      a.u_slice = lv.U;
      a.u_off = u_off;
      a.trace = trace;
      a.log_c = log(0.5 + log(2.0 * (double)lv.N[r] / (delta ? delta[r] : 0.5)));
      a.E = ws.E;
      a.lbt = ws.lbt;
      a.h2 = ws.h2;
      a.rowh2 = ws.rowh2;
      a.rowh2_write = r == 0;
      a.mB = ws.mB;
      a.status = ws.status;
      a.gmask = ws.gmask;
      a.gflag = ws.gflag;
      a.galpha = ws.galpha;
      a.pass_tag = r + 1;
      a.chunk0 = 0;
      a.b0 = 0;
      ok(kh_round(dtype, d, a, S * lv.G[r], ws.e_bytes, r, st));
      u_off += lv.n_r[r] / 2;
      cur = out;
    }
  }
  if (assemble && e == hipSuccess) {
    // after any round the coreset sits n_out apart per slice; with none, the
    // (subsampled or identity) rows n_kept apart
    const int64_t stride = lv.L == 0 ? lv.n_kept : n_out;
    const float lw = (float)log((double)nm / (double)n_out);
    ok(observed(THIN_KERNEL_ASSEMBLE, -1, st, [&] {
      return thin::launch_assemble(S, n, n_sinks, n_out, n_window, cur, stride, idx_out,
                                   logw_out, lw, st);
    }));
  }
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}


}  // namespace

namespace thin {

// thin_compress into a workspace of a fixed size `bytes`: the score region
// takes what the other regions leave (rounds whose buckets do not all fit
// run in several launches).  *need (nullable) receives the bytes the call
// uses; THIN_EWORKSPACE if not even one bucket of every round fits.  With
// workspace == NULL only the arguments' sizes are checked (nothing runs).
int compress_fixed(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H, int64_t n,
                   int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                   int64_t n_uniforms, int32_t* idx_out, void* workspace, size_t bytes,
                   size_t* need, void* stream) {
  int rc = check_shape(B, H, n, d);
  if (rc) return rc;
  Levels lv;
  if (!make_levels(n, n_out, g, &lv) || lv.max_bucket > kMaxBucket) return THIN_EINVAL;
  const int64_t S = B * H;
  // the largest single bucket's scores (0 if every round is local), and
  // every region but the scores
  const size_t one = align256(score_region(S, d, lv, 0));
  const size_t fixed = workspace_size(S, d, lv, 0) - one;
  if (fixed + one > bytes) return THIN_EWORKSPACE;
  const size_t cap = (bytes - fixed) & ~(size_t)255;
  const size_t used = workspace_size(S, d, lv, cap);
  if (used > bytes) return THIN_EWORKSPACE;
  if (need) *need = used;
  if (!workspace) return THIN_OK;
  return compress_impl(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out,
                       workspace, bytes, nullptr, 0, THIN_HALVE_KH, nullptr, 0, 0, nullptr,
                       stream, cap);
}

}  // namespace thin

namespace {

// ---------------------------------------------------------------------------
// Express cache (Alg. 1 with Subsample of Alg. 3 and Compress2 of Alg. 2) and
// Thinformer decoding (Alg. 4, WtdAttention of Alg. 5).  The counters run on
// the host (they depend on the point count and the Subsample draws only); the
// index lists live in the caller's workspace and every Halve call is one KH
// round of a single bucket per slice.
// ---------------------------------------------------------------------------
constexpr int kExMaxL = 30;

// Cor. 2: delta_{m,i} (i >= 0) and delta_m / 2 (i < 0, the Halve phase).
double express_delta(int m, int i, int mbar, double delta) {
  const double dm = 0.5 * delta * (1.0 / log2(m / 2.0 + 2.0) - 1.0 / log2(m / 2.0 + 3.0));
  if (i < 0) return dm / 2.0;
  const int mp = m < mbar ? m : mbar;
  return ldexp(dm, 2 * (i + 1 - mp)) / (3.0 * mp);
}

struct ExLayout {
  size_t status, vmax, E, C[kExMaxL + 1], t1, t2, part, lbt, h2, rowh2, mB, score;
  size_t e_bytes, bytes;
};

ExLayout ex_layout(int64_t S, int64_t d, int64_t n_out, int32_t mbar, int64_t n_max,
                   int64_t kmax) {
  ExLayout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t s4 = (size_t)S * 4;
  L.status = take(4);
  L.vmax = take(s4);
  L.E = take(s4 * 4 * n_out);  // up to 4 n_out before the Halve phase
  for (int i = 0; i <= mbar; ++i) L.C[i] = take(s4 * 2 * n_out);
  L.t1 = take(s4 * 2 * n_out);
  L.t2 = take(s4 * n_out);
  (void)kmax;
  L.part = take(s4 * thin::kDecodeMaxSplit * (d + 2));
  L.lbt = take(s4 * 2 * n_out);
  L.h2 = take(s4 * 2 * n_out);
  L.rowh2 = take(s4 * n_max);
  L.mB = take(s4 * (size_t)((4 * n_out + 63) / 64));
  const size_t per = thin::halve_score_bytes(4 * n_out);
  const size_t all = (size_t)S * per, cap = per > kScoreCap ? per : kScoreCap;
  L.e_bytes = all < cap ? all : cap;
  L.score = take(L.e_bytes);
  L.bytes = off;
  return L;
}

}  // namespace

// Halve calls of a count-only run, for the prefill: the uniform offset of
// every call, by level and Compress2 depth (depth -1: the Halve phase).
struct ExpressCalls {
  std::vector<std::vector<std::vector<int64_t>>> calls;  // [m / 2][depth + 1] -> offsets
  void add(int m, int depth, int64_t u) {
    if ((int)calls.size() <= m / 2) calls.resize(m / 2 + 1);
    auto& lv = calls[m / 2];
    if ((int)lv.size() <= depth + 1) lv.resize(depth + 2);
    lv[depth + 1].push_back(u);
  }
  int64_t count(int m, int depth) const {
    if ((int)calls.size() <= m / 2 || (int)calls[m / 2].size() <= depth + 1) return 0;
    return (int64_t)calls[m / 2][depth + 1].size();
  }
};

struct thin_express {
  int32_t dtype, halve, mbar;
  int64_t B, H, S, d, n_out, n_max, u_slice, kmax;
  double delta;
  unsigned char* ws;
  ExLayout L;
  // Alg. 1 / 2 / 3 counters
  int32_t m, mp;
  int64_t n, ell, nE, upos;
  int64_t nC[kExMaxL + 1];
  int64_t sub_n, sub_i, sub_pos;  // Subsample: points since its reset, the kept one, draws used
  bool over;
  ExpressCalls* rec;  // count-only runs: records every Halve call (nullable)
};

namespace {

template <typename P>
P* ex_ptr(const thin_express* x, size_t off) {
  return reinterpret_cast<P*>(x->ws + off);
}

// Row stride of C_i in the current Compress2: its group size for i < mp, n_out for C_mp.
int64_t ex_stride(const thin_express* x, int i) {
  return i < x->mp ? (x->n_out << (i + 2)) >> x->mp : x->n_out;
}

void ex_reset(thin_express* x) {
  x->mp = x->m < x->mbar ? x->m : x->mbar;
  const int64_t t0 = 4 * x->n_out;  // Compress2's smallest groups: 4 n_out / 2^mp points
  if (x->mp >= 1 && (t0 % ((int64_t)1 << x->mp) != 0 || (t0 >> x->mp) < 2 || ((t0 >> x->mp) & 1)))
    x->over = true;
  for (int i = 0; i <= kExMaxL; ++i) x->nC[i] = 0;
  x->sub_n = 0;
}

// Subsample(m, mbar) needs a draw for the next point (a stratum starts).
bool ex_needs_draw(const thin_express* x) {
  return x->m > x->mbar && (x->sub_n % ((int64_t)1 << (x->m - x->mbar))) == 0;
}

// Subsample(m, mbar).keep for the next point (Alg. 3): above mbar one point
// of every stratum of R = 2^(m - mbar), at offset floor(u R) of its start
// (draws null: u = 0).
bool ex_keep(thin_express* x, const float* draws) {
  x->sub_n += 1;
  if (x->m <= x->mbar) return true;
  const int64_t R = (int64_t)1 << (x->m - x->mbar);
  if ((x->sub_n - 1) % R == 0) {
    const double u = draws ? (double)draws[x->sub_pos] : 0.0;
    x->sub_pos += 1;
    int64_t off = (int64_t)floor(u * (double)R);
    if (off > R - 1) off = R - 1;
    x->sub_i = x->sub_n + off;
  }
  return x->sub_n == x->sub_i;
}

// Device side of one update (null: count only).
struct ExRun {
  const void* K;
  const void* V;
  const float* U;
  uint8_t* trace;
  hipStream_t st;
};

hipError_t ex_halve(thin_express* x, const ExRun* run, const int32_t* in, int64_t N, double delta,
                    int32_t* out, int depth) {
  const int64_t o = x->upos;
  x->upos += N / 2;
  if (!run) {
    if (x->rec) x->rec->add(x->m, depth, o);
    return hipSuccess;
  }
  hipStream_t st = run->st;
  if (x->halve == THIN_HALVE_UNIFORM)
    return observed(THIN_KERNEL_UNIFORM, -1, st, [&] {
      return thin::launch_uniform_halve(x->S, N, in, run->U, x->u_slice, o, out, run->trace, st);
    });
  uint32_t* vmax = ex_ptr<uint32_t>(x, x->L.vmax);
  hipError_t e = observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
    return thin::launch_vmax_rows(x->dtype, run->V, x->n_max, x->d, in, N, N, 1, x->S, vmax, st);
  });
  if (e != hipSuccess) return e;
  thin::HalveArgs a{};
  a.K = run->K;
  a.V = run->V;
  a.n = x->n_max;
  a.ld = x->n_max;
  a.vmax_bits = vmax;
  a.idx_in = in;
  a.n_r = N;
  a.N = (int32_t)N;
  a.G = 1;
  a.S = x->S;
  a.idx_out = out;
  a.U = run->U;
  a.u_slice = x->u_slice;
  a.u_off = o;
  a.trace = run->trace;
  a.log_c = log(0.5 + log(2.0 * (double)N / delta));
  a.E = ex_ptr<float>(x, x->L.score);
  a.lbt = ex_ptr<float>(x, x->L.lbt);
  a.h2 = ex_ptr<float>(x, x->L.h2);
  a.rowh2 = ex_ptr<float>(x, x->L.rowh2);
  a.rowh2_write = 1;
  a.mB = ex_ptr<float>(x, x->L.mB);
  a.status = ex_ptr<int32_t>(x, x->L.status);
  a.chunk0 = 0;
  a.b0 = 0;
  return kh_round(x->dtype, x->d, a, x->S, x->L.e_bytes, -1, st);
}

hipError_t ex_copy(const thin_express* x, const ExRun* run, const int32_t* src, int64_t sstride,
                   int32_t* dst, int64_t dstride, int64_t len) {
  if (!run) return hipSuccess;
  return observed(THIN_KERNEL_EXPRESS, -1, run->st, [&] {
    return thin::launch_rows_copy(src, sstride, dst, dstride, len, x->S, run->st);
  });
}

// Express.update with the next point (Alg. 1), Compress2.update inside (Alg. 2).
// The point itself was already appended, to E (exact phase) or, if Subsample
// keeps it (`keep`), to C_0, by the step's attention launch.
hipError_t ex_update(thin_express* x, const ExRun* run, bool keep) {
  int32_t* E = ex_ptr<int32_t>(x, x->L.E);
  const int64_t sE = 4 * x->n_out;
  hipError_t e = hipSuccess;
  x->n += 1;
  if (x->n <= x->n_out) {  // exact phase
    x->nE += 1;
    return e;
  }
  x->ell += 1;
  if (keep) x->nC[0] += 1;
  int32_t* t1 = ex_ptr<int32_t>(x, x->L.t1);
  for (int i = 0; keep && i < x->mp && e == hipSuccess; ++i) {
    const int64_t T = (x->n_out << (i + 2)) >> x->mp;
    if (x->nC[i] != T) continue;
    const int32_t* in = ex_ptr<int32_t>(x, x->L.C[i]);
    e = ex_halve(x, run, in, T, express_delta(x->m, i, x->mbar, x->delta), t1, i);
    if (e == hipSuccess)
      e = ex_copy(x, run, t1, T / 2, ex_ptr<int32_t>(x, x->L.C[i + 1]) + x->nC[i + 1],
                  ex_stride(x, i + 1), T / 2);
    x->nC[i + 1] += T / 2;
    x->nC[i] = 0;
  }
  if (e == hipSuccess && x->ell == (x->n_out << x->m)) {  // E gets the group's coreset
    e = ex_copy(x, run, ex_ptr<int32_t>(x, x->L.C[x->mp]), ex_stride(x, x->mp), E + x->nE, sE,
                x->nC[x->mp]);
    x->nE += x->nC[x->mp];
    x->ell = 0;
  }
  if (e == hipSuccess && x->n == 4 * (x->n_out << x->m)) {  // Halve phase: E halved twice
    const double dl = express_delta(x->m, -1, x->mbar, x->delta);
    int32_t* t2 = ex_ptr<int32_t>(x, x->L.t2);
    e = ex_halve(x, run, E, x->nE, dl, t1, -1);
    if (e == hipSuccess) e = ex_halve(x, run, t1, x->nE / 2, dl, t2, -1);
    if (e == hipSuccess) e = ex_copy(x, run, t2, x->nE / 4, E, sE, x->nE / 4);
    x->nE /= 4;
    x->m += 2;
  }
  if (x->ell == 0) ex_reset(x);
  return e;
}

// Segments of the weighted cache: C_0, then (self) the point t joining C_0
// with its weight, C_1..C_mp, E.
thin::ExpressSegs ex_segs(const thin_express* x, bool self) {
  thin::ExpressSegs g{};
  const float ln2 = (float)log(2.0);
  g.seg[g.n++] = {ex_ptr<int32_t>(x, x->L.C[0]), ex_stride(x, 0), 0, x->nC[0],
                  -(float)x->mp * ln2};
  if (self) g.seg[g.n++] = {nullptr, 0, x->n, 1, -(float)x->mp * ln2};
  for (int i = 1; i <= x->mp; ++i)
    if (x->nC[i] > 0)
      g.seg[g.n++] = {ex_ptr<int32_t>(x, x->L.C[i]), ex_stride(x, i), 0, x->nC[i],
                      (float)(i - x->mp) * ln2};
  if (x->nE > 0) g.seg[g.n++] = {ex_ptr<int32_t>(x, x->L.E), 4 * x->n_out, 0, x->nE, 0.0f};
  return g;
}

int64_t seg_total(const thin::ExpressSegs& g) {
  int64_t t = 0;
  for (int k = 0; k < g.n; ++k) t += g.seg[k].len;
  return t;
}

// Size checks shared by plan and create; counts uniforms and the largest key
// list over n_max points.
int ex_check(int64_t B, int64_t H, int64_t d, int64_t n_out, int32_t mbar, int64_t n_max,
             int64_t* u_slice, int64_t* kmax, int64_t* draws) {
  if (B < 1 || H < 1 || B * H > kMaxSlices || !supported_d(d)) return THIN_EINVAL;
  if (n_out < 1 || 4 * n_out > kMaxBucket || mbar < 0 || mbar > kExMaxL - 2) return THIN_EINVAL;
  if (n_max < 1 || n_max > kMaxRows) return THIN_EINVAL;
  thin_express x{};
  x.n_out = n_out;
  x.mbar = mbar;
  x.delta = 0.5;
  ex_reset(&x);
  // every stratum keeps its first point (draws of 0): each Halve call comes
  // as early as it can, so the uniforms counted bound those of any draws
  int64_t km = 1;
  for (int64_t t = 0; t < n_max; ++t) {
    if (x.n >= n_out && x.over) return THIN_EINVAL;
    const int64_t k = seg_total(ex_segs(&x, true));
    if (k > km) km = k;
    const bool keep = x.n >= n_out ? ex_keep(&x, nullptr) : true;
    (void)ex_update(&x, nullptr, keep);  // count only: launches nothing
  }
  *u_slice = x.upos;
  *kmax = km;
  *draws = x.sub_pos;
  return THIN_OK;
}
}  // namespace

extern "C" {

int thin_plan(int64_t B, int64_t H, int64_t n, int64_t d, int64_t n_out, int32_t g,
              thin_plan_t* plan) {
  if (!plan) return THIN_EINVAL;
  int rc = check_shape(B, H, n, d);
  if (rc) return rc;
  Levels lv;
  if (!make_levels(n, n_out, g, &lv) || lv.max_bucket > kMaxBucket) return THIN_EINVAL;
  const int64_t S = B * H;
  memset(plan, 0, sizeof(*plan));
  plan->n_kept = lv.n_kept;
  plan->rounds = lv.L;
  plan->compress_levels = lv.mc;
  plan->uniforms_per_slice = lv.U;
  plan->uniforms_total = S * lv.U;
  plan->max_bucket = lv.max_bucket;
  plan->workspace_bytes = workspace_size(S, d, lv);
  return THIN_OK;
}

int thin_compress(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H, int64_t n,
                  int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                  int64_t n_uniforms, int32_t* idx_out, void* workspace,
                  size_t workspace_bytes, void* stream) {
  return compress_impl(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out,
                       workspace, workspace_bytes, nullptr, 0, THIN_HALVE_KH, nullptr, 0, 0,
                       nullptr, stream);
}

int thin_compress_traced(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H,
                         int64_t n, int64_t d, int64_t n_out, int32_t g,
                         const float* uniforms, int64_t n_uniforms, int32_t* idx_out,
                         void* workspace, size_t workspace_bytes, uint8_t* swap_trace,
                         int64_t trace_len, void* stream) {
  if (!swap_trace) return THIN_EINVAL;
  return compress_impl(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out,
                       workspace, workspace_bytes, swap_trace, trace_len, THIN_HALVE_KH, nullptr,
                       0, 0, nullptr, stream);
}

int thin_compress_ex(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H,
                     int64_t n, int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                     int64_t n_uniforms, int32_t* idx_out, void* workspace,
                     size_t workspace_bytes, const thin_compress_opts_t* opts,
                     uint8_t* swap_trace, int64_t trace_len, void* stream) {
  if (!opts) return THIN_EINVAL;
  return compress_impl(K, V, dtype, B, H, n, d, n_out, g, uniforms, n_uniforms, idx_out,
                       workspace, workspace_bytes, swap_trace, trace_len, opts->halve,
                       opts->delta, opts->n_sinks, opts->n_window, opts->logw_out, stream);
}

int thin_attention(const void* Q, const void* K, const void* V, int32_t dtype, int64_t B,
                   int64_t H, int64_t n_q, int64_t n, int64_t d, const int32_t* idx,
                   int64_t n_out, void* O, int32_t out_dtype, void* stream) {
  return thin_attention_ex(Q, K, V, dtype, B, H, n_q, n, d, idx, nullptr, n_out, O, out_dtype,
                           stream);
}

int thin_attention_ex(const void* Q, const void* K, const void* V, int32_t dtype, int64_t B,
                      int64_t H, int64_t n_q, int64_t n, int64_t d, const int32_t* idx,
                      const float* logw, int64_t n_out, void* O, int32_t out_dtype,
                      void* stream) {
  int rc = check_shape(B, H, n, d);
  if (rc) return rc;
  if (n_q < 1 || n_q > kMaxRows || n_out < 1 || n_out > ((int64_t)1 << 30)) return THIN_EINVAL;
  if (dtype != THIN_FP32 && dtype != THIN_BF16) return THIN_EDTYPE;
  if (out_dtype != THIN_FP32 && out_dtype != THIN_BF16) return THIN_EDTYPE;
  if (!Q || !K || !V || !idx || !O) return THIN_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = observed(THIN_KERNEL_ATTENTION, -1, st, [&] {
    return thin::launch_attention(dtype, d, out_dtype, Q, K, V, idx, logw, B * H, n, n_q, n_out,
                                  O, st);
  });
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

int thin_selftest_gram16(int32_t dtype, int64_t d, const void* rows, float* out, void* stream) {
  if (dtype != THIN_FP32 && dtype != THIN_BF16) return THIN_EDTYPE;
  if (!supported_d(d)) return THIN_EINVAL;
  if (!rows || !out) return THIN_EINVAL;
  hipError_t e = thin::launch_gram16(dtype, d, rows, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

int thin_workspace_status(const void* workspace, int32_t* status, void* stream) {
  if (!workspace || !status) return THIN_EINVAL;
  const hipError_t e = hipMemcpyAsync(status, workspace, sizeof(int32_t), hipMemcpyDeviceToHost,
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

int thin_set_launch_hook(thin_launch_hook_t hook, void* ctx) {
  g_hook = hook;
  g_hook_ctx = ctx;
  return THIN_OK;
}

const char* thin_status_str(int status) {
  switch (status) {
    case THIN_OK: return "THIN_OK: success";
    case THIN_EINVAL: return "THIN_EINVAL: invalid size, pointer or level structure";
    case THIN_EDTYPE: return "THIN_EDTYPE: unsupported dtype";
    case THIN_EUNIFORMS: return "THIN_EUNIFORMS: uniforms buffer too short";
    case THIN_EWORKSPACE: return "THIN_EWORKSPACE: workspace missing, too small or misaligned";
    case THIN_EHIP: return "THIN_EHIP: HIP runtime error";
    default: return "THIN: unknown status";
  }
}

}  // extern "C"

namespace {

// ---------------------------------------------------------------------------
// Masked prefill (Alg. 4 for every point of a sequence at once).  A
// count-only run of the Express counters records every Halve call (its
// uniform offset, by level and depth), the kept points and, for every
// point, the cache it attends over.  Then: every Compress2 depth of a level
// is one KH launch over all its calls (per-bucket uniform offsets and
// v_max; every output kept in a node store), the Halve phases run level by
// level, and one launch attends every point over its block's segments plus
// its causal run.
// ---------------------------------------------------------------------------
struct PfLayout {
  int64_t n, n_out, S;
  int32_t mbar;
  int levels;                                  // levels m = 0, 2, .. reached
  std::vector<std::vector<size_t>> region;     // [m/2][depth] node store of the calls
  std::vector<std::vector<int64_t>> rstride;   // [m/2][depth] its row stride per slice
  std::vector<size_t> enode;                   // [m/2] E after the Halve phase of level m - 2
  size_t status, kept, keptrow, keptflag, hp, ein, vmax, absmax, lbt, h2, rowh2, mB, score, utab,
      tiles, segs, c0, w0;
  size_t e_bytes, bytes;
  int64_t max_tiles, max_segs, max_utab;
  size_t tab0;  // the host-built tables occupy [tab0, bytes): one copy from the caller's staging
};

// A run of points attending over one cache (host only): the segments
// [seg0, seg0 + nseg) and C_0 from causal0 with log-weight w0.
struct PfBlock {
  int32_t q0, q1, causal0, seg0, nseg;
  float w0;
};

int64_t group_T(int64_t n_out, int mp, int i) { return (n_out << (i + 2)) >> mp; }

PfLayout pf_layout(int64_t S, int64_t n_out, int32_t mbar, int64_t n, const ExpressCalls& cap) {
  PfLayout L{};
  L.n = n;
  L.n_out = n_out;
  L.S = S;
  L.mbar = mbar;
  L.levels = (int)cap.calls.size();
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t s4 = (size_t)S * 4;
  L.status = take(4);
  L.kept = take(s4 * n);
  L.hp = take(s4 * 2 * n_out);
  L.ein = take(s4 * 4 * n_out);
  L.region.resize(L.levels + 1);
  L.rstride.resize(L.levels + 1);
  L.enode.resize(L.levels + 2);
  int64_t gmax = 1, pmax = 2 * n_out, ucount = 0, bmax = (4 * n_out + 63) / 64;
  for (int lv = 0; lv < L.levels; ++lv) {
    const int m = 2 * lv, mp = m < mbar ? m : mbar;
    L.region[lv].assign(mp, 0);
    L.rstride[lv].assign(mp, 0);
    for (int dd = -1; dd < mp; ++dd) {
      const int64_t c = cap.count(m, dd);
      ucount += c;
      if (dd < 0) continue;
      const int64_t T = group_T(n_out, mp, dd);
      L.rstride[lv][dd] = c * (T / 2) > 0 ? c * (T / 2) : 1;
      L.region[lv][dd] = take(s4 * (size_t)L.rstride[lv][dd]);
      gmax = std::max(gmax, c);
      pmax = std::max(pmax, c * (T / 2));
      bmax = std::max(bmax, c * ((T + 63) / 64));
    }
    L.enode[lv + 1] = take(s4 * n_out);
  }
  L.vmax = take(s4 * gmax);
  L.absmax = take(s4 * n);  // every row's largest |V| entry (the calls' v_max)
  L.lbt = take(s4 * pmax);
  L.h2 = take(s4 * pmax);
  L.rowh2 = take(s4 * n);
  L.mB = take(s4 * (size_t)bmax);
  const size_t per = thin::halve_score_bytes(4 * n_out);
  const size_t all = (size_t)S * per, capb = per > kScoreCap ? per : kScoreCap;
  L.e_bytes = all < capb ? all : capb;
  L.score = take(L.e_bytes);
  // host-built tables: uniform offsets, tiles of 128 points, their cache
  // pieces, every point's C_0 start and log-weight, the kept points
  L.tab0 = off;
  L.max_utab = std::max<int64_t>(ucount, 1);
  L.max_tiles = n / 128 + 2;
  L.max_segs = L.max_tiles * thin::kPrefillMaxSegs;
  L.utab = take(8 * (size_t)L.max_utab);
  L.tiles = take(sizeof(thin::PrefillTile) * (size_t)L.max_tiles);
  L.segs = take(sizeof(thin::PrefillSeg) * (size_t)L.max_segs);
  L.c0 = take(4 * (size_t)n);
  L.w0 = take(4 * (size_t)n);
  L.keptrow = take(4 * (size_t)n);
  L.keptflag = take((size_t)n);
  L.bytes = off;
  return L;
}

// The count-only run of n points: records the calls, the kept points, and,
// given a layout, the blocks of points sharing one cache.
struct PfHost {
  ExpressCalls rec;
  std::vector<int32_t> keptrow;
  std::vector<uint8_t> keptflag;
  std::vector<int64_t> kept_base;  // [m/2]: kept-list index of level m's first point
  std::vector<PfBlock> blocks;
  std::vector<thin::ExpressSeg> segs;
  std::vector<int64_t> piece;  // per segment: the size of its pieces (a call's output, n_out)
  std::vector<thin::PrefillTile> tiles;
  std::vector<thin::PrefillSeg> psegs;
  std::vector<int32_t> c0;
  std::vector<float> w0;
  int64_t query_keys = 0;   // sum over points of the keys each attends over
  int64_t staged_keys = 0;  // sum over 128-point tiles of the keys each stages
};

int pf_run(int64_t n_out, int32_t mbar, int64_t n, const float* draws, int64_t n_draws,
           const PfLayout* L, unsigned char* ws, PfHost* h) {
  thin_express x{};
  x.n_out = n_out;
  x.mbar = mbar;
  x.delta = 0.5;
  x.n_max = n;
  x.rec = &h->rec;
  ex_reset(&x);
  h->keptflag.assign((size_t)n, 0);
  int64_t causal0 = 0;
  std::vector<int64_t> sig, last;
  const float ln2 = (float)log(2.0);
  // without a layout the segments carry no addresses (sizes only)
  auto dev = [&](size_t off) { return L ? reinterpret_cast<int32_t*>(ws + off) : nullptr; };
  auto reg = [&](int lv, int i) -> size_t { return L ? L->region[lv][i] : 0; };
  auto rst = [&](int lv, int i) -> int64_t { return L ? L->rstride[lv][i] : 0; };
  auto eno = [&](int lv) -> size_t { return L ? L->enode[lv] : 0; };
  const size_t kept_off = L ? L->kept : 0;
  for (int64_t p = 0; p < n; ++p) {
    if (x.n >= n_out && x.over) return THIN_EINVAL;
    while ((int64_t)h->kept_base.size() <= x.m / 2) h->kept_base.push_back((int64_t)h->keptrow.size());
    {
      // the cache point p attends over: E (its exact part once complete),
      // C_1..C_mp (outputs of their calls), and C_0 plus p as the causal run
      sig.assign({x.m, x.n >= n_out ? x.nE : -1, causal0});
      for (int i = 1; i <= x.mp; ++i) sig.push_back(x.nC[i]);
      if (p == 0 || sig != last) {
        PfBlock b{};
        b.q0 = (int32_t)p;
        b.causal0 = (int32_t)causal0;
        b.seg0 = (int32_t)h->segs.size();
        b.w0 = -(float)x.mp * ln2;
        const int lv = x.m / 2;
        if (x.n >= n_out) {
          if (x.m == 0) {
            h->segs.push_back({dev(kept_off), n, 0, x.nE, 0.0f});
            h->piece.push_back(n_out);
          } else {
            h->segs.push_back({dev(eno(lv)), n_out, 0, n_out, 0.0f});
            h->piece.push_back(n_out);
            const int64_t gdone = (x.nE - n_out) / n_out;
            if (gdone > 0) {
              h->segs.push_back({dev(reg(lv, x.mp - 1)), rst(lv, x.mp - 1), 0, gdone * n_out,
                                 0.0f});
              h->piece.push_back(n_out);
            }
          }
        }
        for (int i = 1; i <= x.mp; ++i) {
          if (x.nC[i] == 0) continue;
          const int64_t half = group_T(n_out, x.mp, i - 1) / 2;
          const int64_t first = h->rec.count(x.m, i - 1) - x.nC[i] / half;
          int32_t* base = dev(reg(lv, i - 1));
          h->segs.push_back({base ? base + first * half : nullptr, rst(lv, i - 1), 0, x.nC[i],
                             (float)(i - x.mp) * ln2});
          h->piece.push_back(half);
        }
        b.nseg = (int32_t)h->segs.size() - b.seg0;
        if (!h->blocks.empty()) h->blocks.back().q1 = (int32_t)p;
        h->blocks.push_back(b);
        last = sig;
      }
      int64_t fixed = 0;
      for (int k = h->blocks.back().seg0; k < (int)h->segs.size(); ++k) fixed += h->segs[k].len;
      h->query_keys += fixed + (x.n >= n_out ? x.nC[0] : x.n) + 1;
    }
    // Subsample, then the update
    const bool thin_phase = x.n >= n_out;
    if (thin_phase && ex_needs_draw(&x) && draws && x.sub_pos >= n_draws) return THIN_EINVAL;
    const bool keep = thin_phase ? ex_keep(&x, draws) : true;
    h->keptflag[p] = keep ? 1 : 0;
    if (keep) h->keptrow.push_back((int32_t)p);
    const int m_before = x.m;
    const int64_t c0 = h->rec.count(m_before, 0);
    (void)ex_update(&x, nullptr, keep);  // count only: launches nothing
    if (x.n == n_out)
      causal0 = n_out;
    else if (x.n > n_out && (h->rec.count(m_before, 0) != c0 || x.ell == 0))
      causal0 = p + 1;  // C_0 emptied: by Halve_0 or at the end of a group
  }
  if (!h->blocks.empty()) h->blocks.back().q1 = (int32_t)n;
  // tiles of 128 points: the pieces of the blocks a tile overlaps, a piece
  // seen by consecutive blocks kept once with the union of their points
  h->c0.assign((size_t)n, 0);
  h->w0.assign((size_t)n, 0.0f);
  size_t bi = 0;
  for (int64_t t0 = 0; t0 < n; t0 += 128) {
    const int64_t t1 = std::min<int64_t>(t0 + 128, n);
    thin::PrefillTile tl{(int32_t)t0, (int32_t)t1, (int32_t)t1, (int32_t)h->psegs.size(), 0};
    while (bi < h->blocks.size() && h->blocks[bi].q1 <= t0) ++bi;
    for (size_t b = bi; b < h->blocks.size() && h->blocks[b].q0 < t1; ++b) {
      const PfBlock& B = h->blocks[b];
      const int32_t lo = (int32_t)std::max<int64_t>(B.q0, t0), hi = (int32_t)std::min<int64_t>(B.q1, t1);
      for (int32_t p = lo; p < hi; ++p) {
        h->c0[p] = B.causal0;
        h->w0[p] = B.w0;
      }
      tl.causal_lo = std::min(tl.causal_lo, B.causal0);
      for (int k = B.seg0; k < B.seg0 + B.nseg; ++k) {
        const thin::ExpressSeg& g = h->segs[k];
        const int64_t pc = h->piece[k];
        for (int64_t j = 0; j < g.len; j += pc) {
          thin::ExpressSeg a = g;
          if (a.src) a.src += j; else a.start += j;
          a.len = std::min(pc, g.len - j);
          bool merged = false;
          for (size_t q = tl.seg0; q < h->psegs.size(); ++q) {
            thin::PrefillSeg& e = h->psegs[q];
            if (e.g.src == a.src && e.g.start == a.start && e.g.len == a.len &&
                e.g.logw == a.logw && e.g.stride == a.stride && e.vhi == lo) {
              e.vhi = hi;
              merged = true;
              break;
            }
          }
          if (!merged) h->psegs.push_back({a, lo, hi});
        }
      }
    }
    tl.nseg = (int32_t)h->psegs.size() - tl.seg0;
    if (tl.nseg > thin::kPrefillMaxSegs) return THIN_EINVAL;
    int64_t keys = t1 - tl.causal_lo;
    for (int q = tl.seg0; q < tl.seg0 + tl.nseg; ++q) keys += h->psegs[q].g.len;
    h->staged_keys += keys;
    h->tiles.push_back(tl);
  }
  if (L && ((int64_t)h->tiles.size() > L->max_tiles || (int64_t)h->psegs.size() > L->max_segs))
    return THIN_EINVAL;
  // C_0 starts never move back; the prefill kernel turns each causal
  // candidate's visibility into an interval of points on that account
  for (int64_t p = 1; p < n; ++p)
    if (h->c0[p] < h->c0[p - 1]) return THIN_EINVAL;
  return THIN_OK;
}

// The layout and key counts of a prefill depend on its sizes only (the
// Subsample draws move points, not the cache structure), so a count-only run
// per size is kept: a prefill then runs the host counters once, with its
// draws.  (At most kPfCacheMax sizes; the cache is emptied when full.)
struct PfChecked {
  PfLayout L;
  int64_t u_slice, draws, query_keys, staged_keys;
};
constexpr size_t kPfCacheMax = 16;

int pf_check(int64_t B, int64_t H, int64_t n, int64_t d, int64_t n_out, int32_t mbar,
             PfLayout* L, int64_t* u_slice, int64_t* draws, int64_t* query_keys = nullptr,
             int64_t* staged_keys = nullptr) {
  // (a cached entry's arguments all passed the checks below)
  static std::mutex mu;
  static std::map<std::tuple<int64_t, int64_t, int64_t, int64_t, int64_t, int32_t>, PfChecked> cache;
  const auto key = std::make_tuple(B, H, d, n, n_out, mbar);
  {
    std::lock_guard<std::mutex> lock(mu);
    const auto it = cache.find(key);
    if (it != cache.end()) {
      *L = it->second.L;
      *u_slice = it->second.u_slice;
      *draws = it->second.draws;
      if (query_keys) *query_keys = it->second.query_keys;
      if (staged_keys) *staged_keys = it->second.staged_keys;
      return THIN_OK;
    }
  }
  int64_t k = 0;
  const int rc = ex_check(B, H, d, n_out, mbar, n, u_slice, &k, draws);
  if (rc) return rc;
  if (n > ((int64_t)1 << 30)) return THIN_EINVAL;
  PfHost h;
  if (pf_run(n_out, mbar, n, nullptr, 0, nullptr, nullptr, &h)) return THIN_EINVAL;
  *L = pf_layout(B * H, n_out, mbar, n, h.rec);
  if (query_keys) *query_keys = h.query_keys;
  if (staged_keys) *staged_keys = h.staged_keys;
  std::lock_guard<std::mutex> lock(mu);
  if (cache.size() >= kPfCacheMax) cache.clear();
  cache[key] = PfChecked{*L, *u_slice, *draws, h.query_keys, h.staged_keys};
  return THIN_OK;
}

// One batched depth (G calls per slice of N rows each) or a single call.
hipError_t pf_halve(int32_t dtype, int64_t d, int32_t halve, const PfLayout& L,
                    unsigned char* ws, const void* K, const void* V, const float* U,
                    int64_t u_slice, uint8_t* trace, const int32_t* in, int64_t in_stride,
                    int64_t N, int64_t G, const int64_t* u_bucket, int64_t u_off, double delta,
                    int32_t* out, int64_t out_stride, hipStream_t st) {
  const int64_t S = L.S;
  if (halve == THIN_HALVE_UNIFORM)
    return observed(THIN_KERNEL_UNIFORM, -1, st, [&] {
      return thin::launch_uniform_halve(S, G * N, in, U, u_slice, u_off, out, trace, st, N,
                                        u_bucket, in_stride, out_stride);
    });
  uint32_t* vmax = reinterpret_cast<uint32_t*>(ws + L.vmax);
  hipError_t e = observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
    return thin::launch_vmax_table(reinterpret_cast<const uint32_t*>(ws + L.absmax), L.n, in,
                                   in_stride, N, G, S, vmax, st);
  });
  if (e != hipSuccess) return e;
  thin::HalveArgs a{};
  a.K = K;
  a.V = V;
  a.n = L.n;
  a.ld = L.n;
  a.vmax_bits = vmax;
  a.vmax_per_bucket = 1;
  a.idx_in = in;
  a.in_stride = in_stride;
  a.n_r = G * N;
  a.N = (int32_t)N;
  a.G = (int32_t)G;
  a.S = S;
  a.idx_out = out;
  a.out_stride = out_stride;
  a.U = U;
  a.u_slice = u_slice;
  a.u_off = u_off;
  a.u_bucket = u_bucket;
  a.trace = trace;
  a.log_c = log(0.5 + log(2.0 * (double)N / delta));
  a.E = reinterpret_cast<float*>(ws + L.score);
  a.lbt = reinterpret_cast<float*>(ws + L.lbt);
  a.h2 = reinterpret_cast<float*>(ws + L.h2);
  a.rowh2 = reinterpret_cast<float*>(ws + L.rowh2);
  a.rowh2_write = 1;
  a.mB = reinterpret_cast<float*>(ws + L.mB);
  a.status = reinterpret_cast<int32_t*>(ws + L.status);
  if (N <= thin::halve_local_rows(dtype, d))  // every call in one local launch
    return observed(THIN_KERNEL_LOCAL, -1, st,
                    [&] { return thin::launch_local(dtype, d, a, S * G, st); });
  return kh_round(dtype, d, a, S * G, L.e_bytes, -1, st);
}

}  // namespace

extern "C" {

int thin_express_plan(int64_t B, int64_t H, int64_t d, int64_t n_out, int32_t mbar,
                      int64_t n_max, thin_express_plan_t* plan) {
  if (!plan) return THIN_EINVAL;
  int64_t u = 0, k = 0, dr = 0;
  const int rc = ex_check(B, H, d, n_out, mbar, n_max, &u, &k, &dr);
  if (rc) return rc;
  plan->uniforms_per_slice = u;
  plan->max_keys = k;
  plan->subsample_draws = dr;
  plan->workspace_bytes = ex_layout(B * H, d, n_out, mbar, n_max, k).bytes;
  return THIN_OK;
}

int thin_express_create(int32_t dtype, int64_t B, int64_t H, int64_t d, int64_t n_out,
                        int32_t mbar, double delta, int32_t halve, int64_t n_max,
                        void* workspace, size_t workspace_bytes, thin_express_t** out) {
  if (!out) return THIN_EINVAL;
  *out = nullptr;
  if (dtype != THIN_FP32 && dtype != THIN_BF16) return THIN_EDTYPE;
  if (halve != THIN_HALVE_KH && halve != THIN_HALVE_UNIFORM) return THIN_EINVAL;
  if (!(delta > 0.0 && delta < 1.0)) return THIN_EINVAL;
  int64_t u = 0, k = 0, dr = 0;
  const int rc = ex_check(B, H, d, n_out, mbar, n_max, &u, &k, &dr);
  if (rc) return rc;
  const ExLayout L = ex_layout(B * H, d, n_out, mbar, n_max, k);
  if (!workspace || workspace_bytes < L.bytes) return THIN_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return THIN_EWORKSPACE;
  thin_express* x = new (std::nothrow) thin_express();
  if (!x) return THIN_EINVAL;
  x->dtype = dtype;
  x->halve = halve;
  x->mbar = mbar;
  x->B = B;
  x->H = H;
  x->S = B * H;
  x->d = d;
  x->n_out = n_out;
  x->n_max = n_max;
  x->u_slice = u;
  x->kmax = k;
  x->delta = delta;
  x->ws = static_cast<unsigned char*>(workspace);
  x->L = L;
  ex_reset(x);
  *out = x;
  return THIN_OK;
}

int thin_express_step(thin_express_t* x, const void* Q, const void* K, const void* V,
                      const float* uniforms, int64_t n_uniforms, const float* draws,
                      int64_t n_draws, void* O, int32_t out_dtype, uint8_t* swap_trace,
                      void* stream) {
  if (!x || !Q || !K || !V || !O) return THIN_EINVAL;
  if (out_dtype != THIN_FP32 && out_dtype != THIN_BF16) return THIN_EDTYPE;
  if (x->n >= x->n_max || (x->n >= x->n_out && x->over)) return THIN_EINVAL;
  if (x->u_slice > 0 && !uniforms) return THIN_EINVAL;
  if (n_uniforms < x->S * x->u_slice) return THIN_EUNIFORMS;
  const bool thin_phase = x->n >= x->n_out;
  if (thin_phase && ex_needs_draw(x) && (!draws || x->sub_pos >= n_draws)) return THIN_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // WtdAttention: the cache plus the point itself, which joins C_0
  const thin::ExpressSegs g = ex_segs(x, true);
  const int64_t m = seg_total(g);
  // the point enters E (exact phase) or, when Subsample keeps it, C_0
  const bool keep = thin_phase ? ex_keep(x, draws) : true;
  int32_t* app = nullptr;
  int64_t app_stride = 0;
  if (!thin_phase) {
    app = ex_ptr<int32_t>(x, x->L.E) + x->nE;
    app_stride = 4 * x->n_out;
  } else if (keep) {
    app = ex_ptr<int32_t>(x, x->L.C[0]) + x->nC[0];
    app_stride = ex_stride(x, 0);
  }
  const int32_t t = (int32_t)x->n;
  hipError_t e = hipSuccess;
  if (t == 0)  // the status word covers every step since the first
    e = observed(THIN_KERNEL_STATUS, -1, st, [&] {
      return thin::launch_zero_status(ex_ptr<int32_t>(x, x->L.status), st);
    });
  if (e == hipSuccess) e = observed(THIN_KERNEL_ATTENTION, -1, st, [&] {
    return thin::launch_decode_attention(x->dtype, x->d, out_dtype, Q, K, V, g, x->S, x->n_max, m,
                                         ex_ptr<float>(x, x->L.part), O, app, app_stride, t, st);
  });
  const ExRun run{K, V, uniforms, swap_trace, st};
  if (e == hipSuccess) e = ex_update(x, &run, keep);
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

int thin_express_cache(const thin_express_t* x, int32_t* idx, float* logw, int64_t* len,
                       int32_t* m, void* stream) {
  if (!x || !idx || !logw || !len) return THIN_EINVAL;
  const thin::ExpressSegs g = ex_segs(x, false);
  const int64_t k = seg_total(g);
  *len = k;
  if (m) *m = x->m;
  if (k == 0) return THIN_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const hipError_t e = observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
    return thin::launch_express_keys(g, x->S, k, x->kmax, idx, logw, st);
  });
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

int thin_express_next(const thin_express_t* x, int64_t* keys, int64_t* t) {
  if (!x || !keys || !t) return THIN_EINVAL;
  *keys = seg_total(ex_segs(x, true));
  *t = x->n;
  return THIN_OK;
}

int thin_express_destroy(thin_express_t* x) {
  delete x;
  return THIN_OK;
}

}  // extern "C"

extern "C" {

int thin_express_prefill_plan(int64_t B, int64_t H, int64_t n, int64_t d, int64_t n_out,
                              int32_t mbar, thin_prefill_plan_t* plan) {
  if (!plan) return THIN_EINVAL;
  PfLayout L;
  int64_t u = 0, dr = 0, qk = 0, sk = 0;
  const int rc = pf_check(B, H, n, d, n_out, mbar, &L, &u, &dr, &qk, &sk);
  if (rc) return rc;
  plan->uniforms_per_slice = u;
  plan->subsample_draws = dr;
  plan->workspace_bytes = L.bytes;
  plan->attention_keys = qk;
  plan->staged_keys = sk;
  plan->host_staging_bytes = L.bytes - L.tab0;
  return THIN_OK;
}

int thin_express_prefill(int32_t dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                         int64_t n_out, int32_t mbar, double delta, int32_t halve,
                         const void* Q, const void* K, const void* V, const float* uniforms,
                         int64_t n_uniforms, const float* draws, int64_t n_draws, void* O,
                         int32_t out_dtype, void* workspace, size_t workspace_bytes,
                         void* host_staging, size_t host_staging_bytes, uint8_t* swap_trace,
                         void* stream) {
  if (dtype != THIN_FP32 && dtype != THIN_BF16) return THIN_EDTYPE;
  if (out_dtype != THIN_FP32 && out_dtype != THIN_BF16) return THIN_EDTYPE;
  if (halve != THIN_HALVE_KH && halve != THIN_HALVE_UNIFORM) return THIN_EINVAL;
  if (!(delta > 0.0 && delta < 1.0)) return THIN_EINVAL;
  if (!Q || !K || !V || !O) return THIN_EINVAL;
  PfLayout L;
  int64_t u_slice = 0, ndraw = 0;
  int rc = pf_check(B, H, n, d, n_out, mbar, &L, &u_slice, &ndraw);
  if (rc) return rc;
  const int64_t S = B * H;
  if (u_slice > 0 && !uniforms) return THIN_EINVAL;
  if (n_uniforms < S * u_slice) return THIN_EUNIFORMS;
  if (ndraw > 0 && (!draws || n_draws < ndraw)) return THIN_EINVAL;
  if (!workspace || workspace_bytes < L.bytes) return THIN_EWORKSPACE;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return THIN_EWORKSPACE;
  if (!host_staging || host_staging_bytes < L.bytes - L.tab0) return THIN_EWORKSPACE;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  PfHost h;
  rc = pf_run(n_out, mbar, n, draws, n_draws, &L, ws, &h);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // uniform offsets of every call, by level and depth, one table
  std::vector<int64_t> utab;
  std::vector<std::vector<size_t>> uoff(L.levels);
  for (int lv = 0; lv < L.levels && lv < (int)h.rec.calls.size(); ++lv) {
    uoff[lv].assign(h.rec.calls[lv].size(), 0);
    for (size_t k = 0; k < h.rec.calls[lv].size(); ++k) {
      uoff[lv][k] = utab.size();
      utab.insert(utab.end(), h.rec.calls[lv][k].begin(), h.rec.calls[lv][k].end());
    }
  }
  if ((int64_t)utab.size() > L.max_utab) return THIN_EINVAL;
  hipError_t e = hipSuccess;
  auto ok = [&](hipError_t v) {
    if (v != hipSuccess && e == hipSuccess) e = v;
    return e == hipSuccess;
  };
  // the tables are laid out in the caller's staging buffer as in the
  // workspace, then one asynchronous copy moves them (the caller keeps the
  // staging buffer until the stream has passed this call)
  unsigned char* hs = static_cast<unsigned char*>(host_staging);
  auto put = [&](size_t off, const void* src, size_t bytes) {
    if (bytes) memcpy(hs + (off - L.tab0), src, bytes);
  };
  put(L.utab, utab.data(), utab.size() * 8);
  put(L.tiles, h.tiles.data(), h.tiles.size() * sizeof(thin::PrefillTile));
  put(L.segs, h.psegs.data(), h.psegs.size() * sizeof(thin::PrefillSeg));
  put(L.c0, h.c0.data(), h.c0.size() * 4);
  put(L.w0, h.w0.data(), h.w0.size() * 4);
  put(L.keptrow, h.keptrow.data(), h.keptrow.size() * 4);
  put(L.keptflag, h.keptflag.data(), h.keptflag.size());
  ok(hipMemcpyAsync(ws + L.tab0, hs, L.bytes - L.tab0, hipMemcpyHostToDevice, st));
  auto dev = [&](size_t off) { return reinterpret_cast<int32_t*>(ws + off); };
  ok(observed(THIN_KERNEL_STATUS, -1, st,
              [&] { return thin::launch_zero_status(dev(L.status), st); }));
  if (halve == THIN_HALVE_KH)  // the KH calls' v_max come from this table
    ok(observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
      return thin::launch_row_absmax(dtype, V, n, d, S,
                                     reinterpret_cast<uint32_t*>(ws + L.absmax), st);
    }));
  int32_t* kept = dev(L.kept);
  const int64_t nk = (int64_t)h.keptrow.size();
  if (e == hipSuccess && nk > 0)
    ok(observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
      return thin::launch_rows_copy(dev(L.keptrow), 0, kept, n, nk, S, st);
    }));
  const int64_t* ut = reinterpret_cast<const int64_t*>(ws + L.utab);
  // Compress2 of every group: one launch per (level, depth)
  for (int lv = 1; lv < L.levels && e == hipSuccess; ++lv) {
    const int m = 2 * lv, mp = m < mbar ? m : mbar;
    for (int i = 0; i < mp && e == hipSuccess; ++i) {
      const int64_t G = h.rec.count(m, i);
      if (G == 0) break;
      const int64_t T = group_T(n_out, mp, i);
      const int32_t* in = i == 0 ? kept + h.kept_base[lv] : dev(L.region[lv][i - 1]);
      const int64_t in_stride = i == 0 ? n : L.rstride[lv][i - 1];
      ok(pf_halve(dtype, d, halve, L, ws, K, V, uniforms, u_slice, swap_trace, in, in_stride, T,
                  G, ut + uoff[lv][i + 1], 0, express_delta(m, i, mbar, delta),
                  dev(L.region[lv][i]), L.rstride[lv][i], st));
    }
  }
  // Halve phases, level by level: E (the previous Express coreset, then the
  // three groups' coresets) halved twice
  for (int lv = 0; lv < L.levels && e == hipSuccess; ++lv) {
    const int m = 2 * lv, mp = m < mbar ? m : mbar;
    if (h.rec.count(m, -1) < 2) break;
    const double dl = express_delta(m, -1, mbar, delta);
    const int32_t* in = kept;  // level 0: E is the first 4 n_out points
    int64_t in_stride = n;
    if (m > 0) {
      ok(observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
        return thin::launch_rows_copy(dev(L.enode[lv]), n_out, dev(L.ein), 4 * n_out, n_out, S,
                                      st);
      }));
      ok(observed(THIN_KERNEL_EXPRESS, -1, st, [&] {
        return thin::launch_rows_copy(dev(L.region[lv][mp - 1]), L.rstride[lv][mp - 1],
                                      dev(L.ein) + n_out, 4 * n_out, 3 * n_out, S, st);
      }));
      in = dev(L.ein);
      in_stride = 4 * n_out;
    }
    const std::vector<int64_t>& hp = h.rec.calls[lv][0];
    if (e == hipSuccess)
      ok(pf_halve(dtype, d, halve, L, ws, K, V, uniforms, u_slice, swap_trace, in, in_stride,
                  4 * n_out, 1, nullptr, hp[0], dl, dev(L.hp), 2 * n_out, st));
    if (e == hipSuccess)
      ok(pf_halve(dtype, d, halve, L, ws, K, V, uniforms, u_slice, swap_trace, dev(L.hp),
                  2 * n_out, 2 * n_out, 1, nullptr, hp[1], dl, dev(L.enode[lv + 1]), n_out, st));
  }
  if (e == hipSuccess)
    ok(observed(THIN_KERNEL_ATTENTION, -1, st, [&] {
      return thin::launch_prefill_attention(
          dtype, d, out_dtype, Q, K, V, S, n,
          reinterpret_cast<const thin::PrefillTile*>(ws + L.tiles), (int64_t)h.tiles.size(),
          reinterpret_cast<const thin::PrefillSeg*>(ws + L.segs),
          reinterpret_cast<const int32_t*>(ws + L.c0), reinterpret_cast<const float*>(ws + L.w0),
          reinterpret_cast<const uint8_t*>(ws + L.keptflag), O, st);
    }));
  return e == hipSuccess ? THIN_OK : THIN_EHIP;
}

}  // extern "C"
