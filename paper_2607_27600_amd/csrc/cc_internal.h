// Internal declarations shared by the HIP kernels and the C-ABI host code of libcc.
// Device helpers for bf16 storage, CDNA4 MFMA operand types, the KV-cache address
// view, and the launcher entry points each kernel file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cc.h"

namespace cc {

typedef uint16_t u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 2^x on the transcendental unit (v_exp_f32) without the library's denormal fix-up:
// results below 2^-126 flush to zero, which a softmax or log-sum-exp term can afford.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf2f(u16 b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ u16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u16(u >> 16);
}

// Two floats -> packed bf16 pair (lo in bits 0..15), round to nearest even.
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// 32x32x16 bf16 MFMA: A lane l holds row l%32, B lane l holds column l%32; both hold the
// 8 k-slots of lane half l/32.  C lane l holds column l%32, rows 8*(e/4) + 4*(l/32) + e%4.
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Address view of one KV tensor (keys or values) as passed to kernels.
struct KvView {
  const void* base;
  int64_t seq_stride, layer_stride, head_stride, tok_stride, page_stride;
  const int32_t* block_table;
  int32_t page_shift, page_mask, max_pages, pad;
};

template <bool PAGED>
__device__ __forceinline__ int64_t kv_off(const KvView& v, int b, int layer, int h, int t) {
  if constexpr (PAGED) {
    const int page = v.block_table[int64_t(b) * v.max_pages + (t >> v.page_shift)];
    return int64_t(layer) * v.layer_stride + int64_t(page) * v.page_stride +
           int64_t(h) * v.head_stride + int64_t(t & v.page_mask) * v.tok_stride;
  } else {
    return int64_t(b) * v.seq_stride + int64_t(layer) * v.layer_stride +
           int64_t(h) * v.head_stride + int64_t(t) * v.tok_stride;
  }
}

// ------------------------------------------------------------------ launchers
// Each returns hipSuccess or the launch error.  Arguments are validated by the caller.

struct AttnLaunch {
  int dtype;            // cc_dtype
  const void* q;        // [N][Hq][d]
  void* o;              // [N][Hq][d]
  const int32_t* cu_d;  // device cu_seqlens
  const int4* work_d;   // device work list {seq, kv head, row block, 0}; null for one sequence
  int n_work;
  KvView k, v;
  bool paged;
  int layer;
  int n_heads_q, n_heads_kv, head_dim;
  float scale;
  int inclusive;
};
// Rows per attention work item for the given dtype / head_dim.
int attention_rows_per_item(int dtype, int head_dim);
hipError_t launch_attention(const AttnLaunch& a, hipStream_t s);

// GEMM y[M][N] = x[M][K] w[N][K]^T, bf16 in / bf16 out (or f32 for dtype CC_F32).
hipError_t launch_linear(int dtype, const void* x, const void* w, void* y, int M, int N, int K,
                         hipStream_t s);
// out[c][r] = in[r][c], in [rows][cols] (dtype elements).
hipError_t launch_transpose(int dtype, const void* in, void* out, int rows, int cols,
                            hipStream_t s);

// LM head with fused log-sum-exp: per (token, vocab tile) partial (max, sumexp) and the
// target logit, then the combine into scores.
struct LmHeadLaunch {
  int dtype;
  const void* u;        // [N][D]
  const void* w_lm;     // [V][D]
  const int32_t* ids;   // [N]
  float* scores;        // [N]
  float* lse;           // [N] or null
  float2* partial;      // workspace [n_vtiles][N]
  float* target;        // workspace [N]
  const int32_t* cu_d;  // device cu_seqlens
  int n_seqs;
  int N, D, V;
  int n_frozen;
  // bf16 only, optional: the weight packed by launch_pack_rows; u is then packed into
  // u_packed (packed_rows_bytes(N, D)) and the packed kernel runs
  const void* w_packed = nullptr;
  void* u_packed = nullptr;
};
int lmhead_vocab_tile(int dtype);
// Packed operand layout of the LM head (bf16 [rows][cols], cols a multiple of 32): per
// 256-row tile and 32-column step a 16 KB block, the LDS image the kernel stages.
size_t packed_rows_bytes(int64_t rows, int cols);
hipError_t launch_pack_rows(const void* x, int64_t rows, int cols, int64_t ldx, void* out,
                            hipStream_t s);
hipError_t launch_lmhead(const LmHeadLaunch& a, hipStream_t s);

// FP8 LM head: u (dtype) quantized per row into uq / su, then the E4M3 GEMM with the LSE
// epilogue on the scaled logits, the target logits and the combine.
struct LmHeadFp8Launch {
  int dtype;             // of u
  const void* u;         // [N][D]
  const uint8_t* wq;     // [V][D] E4M3 codes
  const float* sw;       // [1] device scale of wq
  const int32_t* ids;    // [N]
  float* scores;         // [N]
  float* lse;            // [N] or null
  uint8_t* uq;           // workspace [N][D]
  float* su;             // workspace [N]
  float* amax_ws;        // workspace [N]
  float2* partial;       // workspace [n_vtiles][N]
  float* target;         // workspace [N]
  const int32_t* cu_d;
  int n_seqs;
  int N, D, V;
  int n_frozen;
};
hipError_t launch_lmhead_fp8(const LmHeadFp8Launch& a, hipStream_t s);
// E4M3 codes and scales of x [rows][cols] (dtype), per row or one for the matrix;
// amax_ws holds rows + 1 floats.
hipError_t launch_quantize_e4m3(int dtype, const void* x, int64_t rows, int cols, int per_row,
                                uint8_t* q, float* scale, float* amax_ws, hipStream_t s);

// Keep selection: one workgroup per segment.
struct SelSeg {
  int64_t start;   // score offset
  int32_t len;
  int32_t k;
  int64_t out;     // keep_idx offset
};
// Up to SEL_INLINE segment descriptors travel by value in the kernel arguments (no upload).
constexpr int SEL_INLINE = 16;
struct SelInline {
  SelSeg s[SEL_INLINE];
  int n;        // descriptors held here (0: all are read from the device table)
  int regular;  // 1: segment b is {start0 + b * stride, len, k, out b * k} (no table)
  int64_t start0, stride;
  int32_t len, k;
};
// True when the segments are equal (length and k) at a fixed start stride with outputs
// back to back: their descriptors need no upload.
bool select_regular(const SelSeg* segs_h, int n_segs);
// segs_h: the descriptors on the host; segs_d: the same in device memory, read only when
// n_segs > SEL_INLINE (may be null otherwise).
hipError_t launch_select(const float* scores, const SelSeg* segs_h, const SelSeg* segs_d,
                         int n_segs, int max_len, int32_t* keep, hipStream_t s);

// KV compaction: one workgroup per (list, layer, head, tensor) plane.
struct CompactPlane {
  int32_t seq, layer, head, list;  // list: index into list table
};
struct CompactList {
  int64_t keep_off;  // offset of the list in keep_idx
  int64_t tok0;      // first row of the sequence in a flat token-major array (0 for caches)
  int32_t k;
  int32_t pad;
};
struct CompactLaunch {
  KvView src[2], dst[2];   // keys, values; strides in BYTES
  int n_tensors;           // 2 (keys and values) or 1
  bool paged;
  int row_bytes;           // head_dim * element size
  const int32_t* keep;
  const CompactList* lists_d;
  const CompactPlane* planes_d;
  int n_planes;            // planes per tensor
  int max_k;               // longest list (bounds the out-of-place grid)
  bool in_place;
  // token/pos ids
  int32_t* ids[2];
  const int32_t* cu_d;
  const int32_t* seq_list_d;  // list index of each sequence's first list
  int n_seqs;
};
hipError_t launch_compact(const CompactLaunch& a, hipStream_t s);

// FULL-mode building blocks (bf16, head_dim 128).
// Split-K: slices a [M][K] x [N][K] product is cut into along K when its 256 x 256 tiles
// would fill under half the chip (1: one pass).  A split product needs a workspace of
// slices * M * N floats for its partial sums.
int gemm_split_slices(int M, int N, int K);
// q[n][:] = RoPE(W_q a[n]) with rot[n][e] = (cos, sin) of the entry's rotation angle.
// part: gemm_split_slices(HD, N, D) * N * HD floats when that count exceeds 1, else unused.
hipError_t launch_qproj_rope(const void* wq, const void* a, void* q, const float2* rot, int N,
                             int D, int HD, float* part, hipStream_t s);
// h[m][:] += x[m][:] W^T (fp32 residual stream).
// part: gemm_split_slices(M, N, K) * M * N floats when that count exceeds 1, else unused.
hipError_t launch_linear_residual(const void* x, const void* w, float* h, int M, int N, int K,
                                  float* part, hipStream_t s);
// act[n][f] = silu(W_gate b[n])[f] * (W_up b[n])[f].
hipError_t launch_gate_up_swiglu(const void* w_gate, const void* w_up, const void* b, void* act,
                                 int N, int D, int F, hipStream_t s);
// h[n][:] = embed[ids[n]][:] (bf16 -> fp32); ids == null widens row n of `embed`.
hipError_t launch_embed(const void* embed, const int32_t* ids, float* h, int N, int D,
                        hipStream_t s);
// y[n][:] = bf16(h[n][:] / sqrt(mean(h[n]^2) + eps) * gamma).
hipError_t launch_rmsnorm(const float* h, const void* gamma, void* y, int N, int D, float eps,
                          hipStream_t s);
// rot[n][e] = (cos, sin)(pos[n] * theta^(-2e/head_dim)), e < head_dim/2, computed in fp64.
// pos == null: positions 0..n_b-1 within each sequence.
hipError_t launch_rope_table(const int32_t* pos, const int32_t* cu, int n_seqs, float2* rot,
                             int N, int head_dim, double theta, hipStream_t s);
}  // namespace cc
