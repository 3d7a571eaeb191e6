// Host-side launchers of the thinning kernels (defined in the .hip files).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace thin {

// One Halve round over buckets b0 .. b0 + nbk - 1 (bucket = slice * G + t).
struct HalveArgs {
  const void* K;
  const void* V;
  int64_t n;                  // thinned rows per slice
  int64_t ld;                 // rows between consecutive slices of K/V (>= n)
  const uint32_t* vmax_bits;  // [S] bit pattern of v_max (non-negative float)
  const int32_t* idx_in;      // [S, n_r] rows entering this round, or null = identity
  int64_t n_r;                // rows per slice entering this round
  int32_t N;                  // bucket size (even, >= 2)
  int32_t G;                  // buckets per slice
  int64_t S;                  // slices
  int32_t* idx_out;           // [S, n_r / 2]
  const float* U;             // uniforms
  int64_t u_slice;            // uniforms per slice
  int64_t u_off;              // offset of this round's draws within a slice
  uint8_t* trace;             // nullable, indexed like U
  double log_c;               // log(1/2 + log(2N/delta))
  float* E;                   // pair scores of the launched buckets (halve_score_bytes each)
  float* lbt;                 // [S, n_r / 2] scaled log b per pair
  float* h2;                  // [S, n_r / 2] scale exponent per pair
  int64_t b0;                 // first bucket of this launch
  int64_t e_tiles;            // score tiles per bucket (set by launch_scores)
  int32_t ch;                 // column tiles per score workgroup (set by launch_scores)
  float* rowh2;               // [S, n] scale exponent of every row, written by the first round
  int32_t rowh2_write;        // this round writes rowh2 (and reads it only after writing)
  int32_t chunk0;             // first column chunk of a score launch (set by launch_scores)
  int32_t nz;                 // column chunks per group in a score launch (set by launch_scores)
  int32_t ngrp;               // row groups per bucket (set by launch_scores)
  int64_t nbk;                // buckets of a score launch (set by launch_scores)
  int32_t ipb;                // score workgroups per bucket in a launch (set by launch_scores)
  int32_t il;                 // buckets interleaved per XCD in a score launch (set by launch_scores)
  // Optional (zero / null: the packed layout above)
  const int64_t* u_bucket;    // [G] first uniform of bucket t within its slice (else u_off + t*N/2)
  int32_t vmax_per_bucket;    // vmax_bits indexed by bucket (s * G + t) instead of slice
  int64_t in_stride;          // idx_in row stride per slice (0: n_r)
  int64_t out_stride;         // idx_out row stride per slice (0: n_r / 2)
  // Required by the two-launch path
  float* mB;                  // [buckets, ceil(N / 64)] largest row scale of every 64-row block
  int32_t* status;            // nullable: set nonzero if a bounded wait of the decisions gave up
  // Decision helpers (gmask null: none).  A round that runs as one launch may
  // spread each bucket's bulk sums over helper workgroups on other compute
  // units: the bucket's workgroup publishes every block's decisions in gmask,
  // helpers add the early rows of a chunk of pairs and hand over the partial
  // alpha in galpha (gflag marks it ready).  gmask and gflag hold zero or
  // values of earlier rounds of the same call (their tags differ).
  uint64_t* gmask;            // [nbk, nblk] (tag(round, block) << 32) | decisions
  uint32_t* gflag;            // [nbk, nch] round tag once the chunk's partial is written
  uint64_t* galpha;           // [nbk, N / 2] partial alpha of every pair (float64 bits)
  int32_t pass_tag;           // round tag, nonzero and distinct per round of a call
  int32_t pass_h;             // helper workgroups per bucket (set by launch_decide)
};

// Device status word (the first word of every workspace): 0 = every bounded
// wait of the call's decision passes completed.
constexpr int32_t kStatusWaitExhausted = 1;

// thin_compress (KH, no trace) into a workspace of exactly `bytes` (api.cpp):
// the score region takes what the other regions leave.  workspace == NULL:
// validation only.  *need receives the bytes used.  Returns a thin_status_t.
int compress_fixed(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H, int64_t n,
                   int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                   int64_t n_uniforms, int32_t* idx_out, void* workspace, size_t bytes,
                   size_t* need, void* stream);

// dtype: 0 = fp32, 1 = bf16.  Returns a hipError_t.
// v_max of n rows per slice, slices ld rows apart.
// status (nullable) is cleared by the same launch, and max(S, zero_words)
// words from vmax_bits on (the decision helpers' flags follow the bits).
hipError_t launch_vmax(int dtype, const void* V, int64_t S, int64_t n, int64_t ld, int64_t d,
                       uint32_t* vmax_bits, hipStream_t st, int32_t* status = nullptr,
                       int64_t zero_words = 0);
hipError_t launch_zero_status(int32_t* status, hipStream_t st);
hipError_t launch_subsample(int64_t S, int64_t n, int64_t n_kept, const float* U,
                            int64_t u_slice, int32_t* idx0, hipStream_t st);
hipError_t launch_fill_rows(int64_t S, int64_t n_out, const int32_t* src, int64_t src_stride,
                            int32_t* dst, hipStream_t st);
hipError_t launch_zero_u8(uint8_t* p, int64_t count, hipStream_t st);
// idx [S, ns + n_out + nw] = sinks, ns + coreset (src, stride src_stride; null =
// identity), window rows of an n-row slice; logw (nullable) 0 or lw_core.
hipError_t launch_assemble(int64_t S, int64_t n, int64_t ns, int64_t n_out, int64_t nw,
                           const int32_t* src, int64_t src_stride, int32_t* dst, float* logw,
                           float lw_core, hipStream_t st);
// One round of uniform halving of every slice: pair p of a slice keeps row
// 2p+1 of the round's input iff its uniform is below 1/2.
hipError_t launch_uniform_halve(int64_t S, int64_t n_r, const int32_t* idx_in, const float* U,
                                int64_t u_slice, int64_t u_off, int32_t* idx_out,
                                uint8_t* trace, hipStream_t st, int64_t N = 0,
                                const int64_t* u_bucket = nullptr, int64_t in_stride = 0,
                                int64_t out_stride = 0);
// Every round of uniform halving in one launch (one workgroup per slice,
// indices in LDS); only for n_kept <= 32768 (uniform_fused_ok).
bool uniform_fused_ok(int64_t n_kept);
hipError_t launch_uniform_compress(int64_t S, int64_t n_kept, int32_t L, const int32_t* idx0,
                                   const float* U, int64_t u_slice, int64_t u_off0,
                                   int32_t* idx_out, int64_t n_out, uint8_t* trace,
                                   hipStream_t st);
// Score tiles and score bytes of one N-row bucket (64-row decision blocks).
int64_t halve_score_tiles(int64_t N);
size_t halve_score_bytes(int64_t N);
// Pair scores, then the decision pass, for nbk buckets starting at a.b0.
hipError_t launch_scores(int dtype, int64_t d, const HalveArgs& a, int64_t nbk, hipStream_t st);
hipError_t launch_decide(const HalveArgs& a, int64_t nbk, hipStream_t st);
// Decision helpers (HalveArgs.gmask): eligible rounds and the most helpers.
constexpr int64_t kHelperMaxBuckets = 128;
constexpr int64_t kHelperMinPairs = 2048;
constexpr int kMaxHelpers = 7;
// Buckets of at most halve_local_rows(dtype, d) rows: the whole round (scores
// in LDS, then the decisions) in one launch, no score buffer.
int64_t halve_local_rows(int dtype, int64_t d);
hipError_t launch_local(int dtype, int64_t d, const HalveArgs& a, int64_t nbk, hipStream_t st);

// Express cache (express.hip).  A segment of a slice's key list: src null =
// the rows start .. start+len-1, else src[s * stride + 0 .. len-1]; every key
// of the segment has log-weight logw.
struct ExpressSeg {
  const int32_t* src;
  int64_t stride;
  int64_t start;
  int64_t len;
  float logw;
};
constexpr int kExpressMaxSegs = 34;
struct ExpressSegs {
  ExpressSeg seg[kExpressMaxSegs];
  int n;
};
hipError_t launch_rows_copy(const int32_t* src, int64_t src_stride, int32_t* dst,
                            int64_t dst_stride, int64_t len, int64_t S, hipStream_t st);
// v_max bits of G calls per slice, call t over the rows idx[s * in_stride +
// t * N + 0..N) of V (slices ld rows apart), into vmax_bits[s * G + t].
hipError_t launch_vmax_rows(int dtype, const void* V, int64_t ld, int64_t d, const int32_t* idx,
                            int64_t in_stride, int64_t N, int64_t G, int64_t S,
                            uint32_t* vmax_bits, hipStream_t st);
// The largest |V| entry of every row of S slices of n rows (V [S, n, d]),
// float bits at absmax[s * n + r]; then the v_max of G calls per slice from
// that table (calls as in launch_vmax_rows), equal to launch_vmax_rows'.
hipError_t launch_row_absmax(int dtype, const void* V, int64_t n, int64_t d, int64_t S,
                             uint32_t* absmax, hipStream_t st);
hipError_t launch_vmax_table(const uint32_t* absmax, int64_t n, const int32_t* idx,
                             int64_t in_stride, int64_t N, int64_t G, int64_t S,
                             uint32_t* vmax_bits, hipStream_t st);
// idx / logw [S, out_stride]: the segments laid out one after another in the
// first m entries of each slice (their lengths sum to m).
hipError_t launch_express_keys(const ExpressSegs& segs, int64_t S, int64_t m, int64_t out_stride,
                               int32_t* idx, float* logw, hipStream_t st);
// Weighted attention of one query per slice (Q [S, d], O [S, d]) over the m
// keys of the segments (rows of K / V, slices ld rows apart): the keys of a
// slice split over decode_attention_split(m) workgroups; with one, it writes
// the output itself, else a second launch merges their partials (S * split *
// (d + 2) floats in `part`).  The last launch also writes app_val to
// app[s * app_stride] when app is non-null.
#ifndef DEC_KPG
#define DEC_KPG 1024
#endif
constexpr int kDecodeKeysPerGroup = DEC_KPG;
constexpr int kDecodeMaxSplit = 16;
int decode_attention_split(int64_t m);
hipError_t launch_decode_attention(int dtype, int64_t d, int out_dtype, const void* Q,
                                   const void* K, const void* V, const ExpressSegs& segs,
                                   int64_t S, int64_t ld, int64_t m, float* part, void* O,
                                   int32_t* app, int64_t app_stride, int32_t app_val,
                                   hipStream_t st);


// Masked prefill over the Express cache: a tile is the points [q0, q1) (at
// most 128); its keys are the pieces [seg0, seg0 + nseg) (at most 256), piece
// k seen by the points vlo..vhi-1, then the causal candidates causal_lo ..
// q1-1, candidate r seen by point p iff r == p, or kept[r] and
// c0[p] <= r < p, with p's C_0 log-weight w0[p].
struct PrefillTile {
  int32_t q0, q1, causal_lo, seg0, nseg;
};
struct PrefillSeg {
  ExpressSeg g;
  int32_t vlo, vhi;
};
constexpr int kPrefillMaxSegs = 256;
hipError_t launch_prefill_attention(int dtype, int64_t d, int out_dtype, const void* Q,
                                    const void* K, const void* V, int64_t S, int64_t n,
                                    const PrefillTile* tiles, int64_t ntiles,
                                    const PrefillSeg* segs, const int32_t* c0, const float* w0,
                                    const uint8_t* kept, void* O, hipStream_t st);

// logw (nullable) [S, n_out]: log-weight of every coreset key.
hipError_t launch_attention(int dtype, int64_t d, int out_dtype, const void* Q, const void* K,
                            const void* V, const int32_t* idx, const float* logw, int64_t S,
                            int64_t n, int64_t n_q, int64_t n_out, void* O, hipStream_t st);

hipError_t launch_gram16(int dtype, int64_t d, const void* rows, float* out, hipStream_t st);

}  // namespace thin
