// C ABI of libcc: argument validation, planning (grids, work lists, workspace layout)
// and kernel launches for the refresh-scoring pass.  Host code only; every kernel lives
// in its own translation unit behind the launchers declared in cc_internal.h.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "cc_internal.h"

using namespace cc;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }
int esize(int dtype) { return dtype == CC_BF16 ? 2 : 4; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

#define CC_TRY(x)                       \
  do {                                  \
    cc_status _st = (x);                \
    if (_st != CC_OK) return _st;       \
  } while (0)

#define CC_HIP(x)                                   \
  do {                                              \
    if ((x) != hipSuccess) return CC_ERR_HIP;       \
  } while (0)

cc_status check_problem(const cc_problem* p) {
  if (!p) return CC_ERR_ARG;
  if (p->dtype != CC_F32 && p->dtype != CC_BF16) return CC_ERR_DTYPE;
  if (p->mode != CC_MODE_LAST_LAYER && p->mode != CC_MODE_FULL &&
      p->mode != CC_MODE_LAST_LAYER_H && p->mode != CC_MODE_LAST_LAYER_FUSED)
    return CC_ERR_ARG;
  if (p->diag != CC_DIAG_STRICT && p->diag != CC_DIAG_INCLUSIVE) return CC_ERR_ARG;
  if (p->n_seqs < 1 || !p->cu_seqlens_h || !p->cu_seqlens_d) return CC_ERR_ARG;
  if (p->cu_seqlens_h[0] != 0) return CC_ERR_SHAPE;
  for (int b = 0; b < p->n_seqs; ++b)
    if (p->cu_seqlens_h[b + 1] < p->cu_seqlens_h[b]) return CC_ERR_SHAPE;
  if (p->n_heads_q < 1 || p->n_heads_kv < 1) return CC_ERR_SHAPE;
  if (p->n_heads_q % p->n_heads_kv != 0) return CC_ERR_SHAPE;
  if (p->head_dim < 1 || p->hidden < 1 || p->vocab < 1) return CC_ERR_SHAPE;
  if (p->n_frozen < 0) return CC_ERR_ARG;
  if (!std::isfinite(p->softmax_scale) || p->softmax_scale < 0.f) return CC_ERR_ARG;
  if (p->head_dim != 64 && p->head_dim != 128) return CC_ERR_UNSUPPORTED;
  // bf16 projections and the LM head step K in 64-element tiles
  if (p->dtype == CC_BF16 && p->hidden % 64 != 0) return CC_ERR_UNSUPPORTED;
  if (p->mode == CC_MODE_FULL || p->mode == CC_MODE_LAST_LAYER_H) {
    if ((p->mode == CC_MODE_FULL && p->n_layers < 1) || p->ffn < 1) return CC_ERR_SHAPE;
    if (p->dtype != CC_BF16) return CC_ERR_UNSUPPORTED;
    // the W_q epilogue applies RoPE with one wave's 128 rows spanning exactly one head
    if (p->head_dim != 128) return CC_ERR_UNSUPPORTED;
    if (p->ffn % 64 != 0) return CC_ERR_UNSUPPORTED;
    if (!(p->rope_theta > 0.f) || !(p->rms_eps >= 0.f)) return CC_ERR_ARG;
  }
  if (p->lmhead_packed != 0 && p->lmhead_packed != 1) return CC_ERR_ARG;
  if (p->lmhead_packed && p->dtype != CC_BF16) return CC_ERR_UNSUPPORTED;
  return CC_OK;
}

int n_tokens(const cc_problem* p) { return p->cu_seqlens_h[p->n_seqs]; }
int max_len(const cc_problem* p) {
  int m = 0;
  for (int b = 0; b < p->n_seqs; ++b) m = std::max(m, p->cu_seqlens_h[b + 1] - p->cu_seqlens_h[b]);
  return m;
}

cc_status check_kv(const cc_problem* p, const cc_kv* kv, int min_layers) {
  if (!kv || !kv->k || !kv->v) return CC_ERR_ARG;
  if (kv->layout != CC_KV_CONTIGUOUS && kv->layout != CC_KV_PAGED) return CC_ERR_ARG;
  if (kv->n_layers < min_layers) return CC_ERR_SHAPE;
  if (kv->layer_stride < 0 || kv->head_stride < 0 || kv->tok_stride < p->head_dim)
    return CC_ERR_SHAPE;
  const int es = esize(p->dtype);
  if (!aligned16(kv->k) || !aligned16(kv->v)) return CC_ERR_ARG;
  auto str_ok = [&](int64_t s) { return (s * es) % 16 == 0; };
  if (!str_ok(kv->layer_stride) || !str_ok(kv->head_stride) || !str_ok(kv->tok_stride))
    return CC_ERR_UNSUPPORTED;
  if (kv->layout == CC_KV_PAGED) {
    if (!kv->block_table || !is_pow2(kv->page_size) || kv->page_size < 16) return CC_ERR_ARG;
    if (kv->page_stride < 0 || !str_ok(kv->page_stride)) return CC_ERR_UNSUPPORTED;
    // in-page byte offsets are 32-bit in the kernels
    constexpr int64_t kPageLimit = int64_t(1) << 32;
    if (kv->page_stride * es >= kPageLimit || int64_t(kv->page_size) * kv->tok_stride * es >= kPageLimit)
      return CC_ERR_UNSUPPORTED;
    const int need = (max_len(p) + kv->page_size - 1) / kv->page_size;
    if (kv->max_pages < need) return CC_ERR_SHAPE;
  } else {
    if (kv->seq_stride < 0 || !str_ok(kv->seq_stride)) return CC_ERR_UNSUPPORTED;
  }
  return CC_OK;
}

// Address view for kernels; byte_strides = true multiplies strides by the element size.
KvView make_view(const cc_kv* kv, const void* base, int es_mult) {
  KvView v;
  v.base = base;
  v.seq_stride = kv->seq_stride * es_mult;
  v.layer_stride = kv->layer_stride * es_mult;
  v.head_stride = kv->head_stride * es_mult;
  v.tok_stride = kv->tok_stride * es_mult;
  v.page_stride = kv->page_stride * es_mult;
  v.block_table = kv->block_table;
  int shift = 0;
  if (kv->layout == CC_KV_PAGED)
    while ((1 << shift) < kv->page_size) ++shift;
  v.page_shift = shift;
  v.page_mask = kv->layout == CC_KV_PAGED ? kv->page_size - 1 : 0;
  v.max_pages = kv->max_pages;
  v.pad = 0;
  return v;
}

float softmax_scale(const cc_problem* p) {
  return p->softmax_scale > 0.f ? p->softmax_scale : 1.f / std::sqrt(float(p->head_dim));
}

// Attention work items, heaviest first: an item's cost is the number of keys its first
// row may attend to, n_b - first position.
std::vector<int4> attention_work(const cc_problem* p) {
  const int rows_item = attention_rows_per_item(p->dtype, p->head_dim);
  const int g = p->n_heads_q / p->n_heads_kv;
  std::vector<int4> items;
  std::vector<int64_t> cost;
  for (int b = 0; b < p->n_seqs; ++b) {
    const int n = p->cu_seqlens_h[b + 1] - p->cu_seqlens_h[b];
    const int64_t rows = int64_t(n) * g;
    const int nrb = int((rows + rows_item - 1) / rows_item);
    for (int rb = 0; rb < nrb; ++rb)
      for (int h = 0; h < p->n_heads_kv; ++h) {
        items.push_back(make_int4(b, h, rb, 0));
        cost.push_back(n - int64_t(rb) * rows_item / g);
      }
  }
  std::vector<int> idx(items.size());
  for (size_t i = 0; i < idx.size(); ++i) idx[i] = int(i);
  std::stable_sort(idx.begin(), idx.end(), [&](int a, int c) { return cost[a] > cost[c]; });
  std::vector<int4> out(items.size());
  for (size_t i = 0; i < idx.size(); ++i) out[i] = items[idx[i]];
  return out;
}

size_t attention_ws_bytes(const cc_problem* p) {
  const int rows_item = attention_rows_per_item(p->dtype, p->head_dim);
  const int g = p->n_heads_q / p->n_heads_kv;
  size_t items = 0;
  for (int b = 0; b < p->n_seqs; ++b) {
    const int64_t n = p->cu_seqlens_h[b + 1] - p->cu_seqlens_h[b];
    items += size_t((n * g + rows_item - 1) / rows_item) * p->n_heads_kv;
  }
  return align_up(items * sizeof(int4));
}

// Input width of the LM head: the model width, or Hq*d for the W_o-folded weight.
int lmhead_k(const cc_problem* p) {
  return p->mode == CC_MODE_LAST_LAYER_FUSED ? p->n_heads_q * p->head_dim : p->hidden;
}

// LM-head workspace: per-(vocabulary tile, entry) partials, target logits and, for the
// packed LM head, the packed input rows.
size_t lmhead_ws_bytes(const cc_problem* p) {
  const size_t N = n_tokens(p);
  const int vt = lmhead_vocab_tile(p->dtype);
  const size_t n_vt = (p->vocab + vt - 1) / vt;
  size_t b = align_up(n_vt * N * sizeof(float2)) + align_up(N * sizeof(float));
  if (p->lmhead_packed) b += align_up(packed_rows_bytes(int64_t(N), lmhead_k(p)));
  return b;
}

struct ScoreLayout {
  size_t attn, o, u, lm, total;
};

struct FullLayout {
  size_t attn, rot, h, a, q, o, act, lm, part, total;
};

FullLayout full_layout(const cc_problem* p) {
  FullLayout L;
  const size_t N = n_tokens(p);
  const size_t HD = size_t(p->n_heads_q) * p->head_dim;
  size_t off = 0;
  L.attn = off;
  off += attention_ws_bytes(p);
  L.rot = off;
  off += align_up(N * (p->head_dim / 2) * sizeof(float2));
  L.h = off;
  off += align_up(N * p->hidden * sizeof(float));
  L.a = off;
  off += align_up(N * p->hidden * 2);
  L.q = off;
  off += align_up(N * HD * 2);
  L.o = off;
  off += align_up(N * HD * 2);
  L.act = off;
  off += align_up(N * size_t(p->ffn) * 2);
  L.lm = off;
  off += lmhead_ws_bytes(p);
  // split-K partial sums of the projections whose tiles underfill the chip (small N)
  const int D = p->hidden, F = p->ffn, hd = int(HD);
  size_t part = 0;
  auto need = [&](int M, int Nn, int K) {
    const int S = gemm_split_slices(M, Nn, K);
    if (S > 1) part = std::max(part, size_t(S) * size_t(M) * size_t(Nn) * sizeof(float));
  };
  need(hd, int(N), D);   // W_q
  need(int(N), D, hd);   // W_o
  need(int(N), D, F);    // W_down
  L.part = off;
  off += align_up(part);
  L.total = off;
  return L;
}

ScoreLayout score_layout(const cc_problem* p) {
  ScoreLayout L;
  const size_t N = n_tokens(p), es = esize(p->dtype);
  size_t off = 0;
  L.attn = off;
  off += attention_ws_bytes(p);
  L.o = off;
  off += align_up(N * p->n_heads_q * p->head_dim * es);
  L.u = off;
  if (p->mode != CC_MODE_LAST_LAYER_FUSED) off += align_up(N * p->hidden * es);
  L.lm = off;
  off += lmhead_ws_bytes(p);
  L.total = off;
  return L;
}

char* at(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

// Attention over cache layer `layer`.  The work list is uploaded into `ws` unless an earlier
// call of the same cc_score already did (upload = false).
cc_status run_attention(const cc_problem* p, const void* q, const cc_kv* kv, int layer, void* o,
                        void* ws, hipStream_t s, bool upload = true) {
  std::vector<int4> work = attention_work(p);
  if (work.empty()) return CC_OK;
  // one sequence: the kernel derives each item from its block index, nothing is uploaded
  const bool table = p->n_seqs > 1;
  if (upload && table)
    CC_HIP(hipMemcpyAsync(ws, work.data(), work.size() * sizeof(int4), hipMemcpyHostToDevice, s));
  AttnLaunch a;
  a.dtype = p->dtype;
  a.q = q;
  a.o = o;
  a.cu_d = p->cu_seqlens_d;
  a.work_d = table ? static_cast<const int4*>(ws) : nullptr;
  a.n_work = int(work.size());
  a.k = make_view(kv, kv->k, 1);
  a.v = make_view(kv, kv->v, 1);
  a.paged = kv->layout == CC_KV_PAGED;
  a.layer = layer;
  a.n_heads_q = p->n_heads_q;
  a.n_heads_kv = p->n_heads_kv;
  a.head_dim = p->head_dim;
  a.scale = softmax_scale(p);
  a.inclusive = p->diag == CC_DIAG_INCLUSIVE;
  CC_HIP(launch_attention(a, s));
  return CC_OK;
}

// LM head over rows u [N][D]; D is the model width unless given (the fused weight's
// input width Hq*d).
cc_status run_lmhead(const cc_problem* p, const void* u, const void* w_lm, const int32_t* ids,
                     float* scores, float* lse, void* ws, hipStream_t s, int D = 0,
                     const void* w_packed = nullptr) {
  const int N = n_tokens(p);
  const int vt = lmhead_vocab_tile(p->dtype);
  const size_t n_vt = (p->vocab + vt - 1) / vt;
  LmHeadLaunch a;
  a.dtype = p->dtype;
  a.u = u;
  a.w_lm = w_lm;
  a.ids = ids;
  a.scores = scores;
  a.lse = lse;
  a.partial = reinterpret_cast<float2*>(ws);
  a.target = reinterpret_cast<float*>(at(ws, align_up(n_vt * N * sizeof(float2))));
  a.cu_d = p->cu_seqlens_d;
  a.n_seqs = p->n_seqs;
  a.N = N;
  a.D = D > 0 ? D : p->hidden;
  a.V = p->vocab;
  a.n_frozen = p->n_frozen;
  if (p->lmhead_packed) {
    if (!w_packed) return CC_ERR_ARG;
    a.w_packed = w_packed;
    a.u_packed = at(ws, align_up(n_vt * N * sizeof(float2)) + align_up(N * sizeof(float)));
  }
  CC_HIP(launch_lmhead(a, s));
  return CC_OK;
}

// The row-major LM head weight, needed unless the packed one is used.
bool lm_weight_ok(const cc_problem* p, const void* w_lm) {
  return p->lmhead_packed || (w_lm && aligned16(w_lm));
}

// The packed LM head needs its weight (checked before anything is launched).
cc_status check_packed(const cc_problem* p, const void* w_packed) {
  if (!p->lmhead_packed || n_tokens(p) == 0) return CC_OK;
  if (!w_packed || !aligned16(w_packed)) return CC_ERR_ARG;
  return CC_OK;
}

cc_status check_ws(void* ws, size_t have, size_t need) {
  if (have < need) return CC_ERR_WORKSPACE;
  if (need > 0 && !ws) return CC_ERR_ARG;
  if (need > 0 && (reinterpret_cast<uintptr_t>(ws) % kAlign) != 0) return CC_ERR_ARG;
  return CC_OK;
}

// Full L-layer pass (Sec. 3.1): h = E[x]; per layer a = RMSNorm(h), q = RoPE(W_q a),
// o = counter-causal attention on the stored K_l, V_l, h += W_o o, b = RMSNorm(h),
// h += W_down (silu(W_gate b) * W_up b); then u = RMSNorm(h) and the LM head.
cc_status score_full(const cc_problem* p, const cc_inputs* in, float* scores, void* ws,
                     size_t ws_bytes, void* stream) {
  CC_TRY(check_kv(p, &in->kv, p->n_layers));
  const int N = n_tokens(p);
  if (N > 0 && (!in->embed || !in->layers_h || !in->final_norm || !in->token_ids || !scores))
    return CC_ERR_ARG;
  if (N > 0) {
    if (!aligned16(in->embed) || !lm_weight_ok(p, in->w_lm) || !aligned16(in->final_norm))
      return CC_ERR_ARG;
    for (int l = 0; l < p->n_layers; ++l) {
      const cc_layer_weights& W = in->layers_h[l];
      const void* ptrs[7] = {W.attn_norm, W.wq, W.wo, W.mlp_norm, W.w_gate, W.w_up, W.w_down};
      for (const void* q : ptrs)
        if (!q || !aligned16(q)) return CC_ERR_ARG;
    }
  }
  CC_TRY(check_packed(p, in->w_lm_packed));
  const FullLayout L = full_layout(p);
  CC_TRY(check_ws(ws, ws_bytes, L.total));
  if (N == 0) return CC_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int D = p->hidden, F = p->ffn, HD = p->n_heads_q * p->head_dim;
  float2* rot = reinterpret_cast<float2*>(at(ws, L.rot));
  float* h = reinterpret_cast<float*>(at(ws, L.h));
  void* a = at(ws, L.a);
  void* q = at(ws, L.q);
  void* o = at(ws, L.o);
  void* act = at(ws, L.act);
  float* part = reinterpret_cast<float*>(at(ws, L.part));
  CC_HIP(launch_rope_table(in->pos_ids, p->cu_seqlens_d, p->n_seqs, rot, N, p->head_dim,
                           double(p->rope_theta), s));
  CC_HIP(launch_embed(in->embed, in->token_ids, h, N, D, s));
  for (int l = 0; l < p->n_layers; ++l) {
    const cc_layer_weights& W = in->layers_h[l];
    CC_HIP(launch_rmsnorm(h, W.attn_norm, a, N, D, p->rms_eps, s));
    CC_HIP(launch_qproj_rope(W.wq, a, q, rot, N, D, HD, part, s));
    CC_TRY(run_attention(p, q, &in->kv, l, o, at(ws, L.attn), s, l == 0));
    CC_HIP(launch_linear_residual(o, W.wo, h, N, D, HD, part, s));
    CC_HIP(launch_rmsnorm(h, W.mlp_norm, a, N, D, p->rms_eps, s));
    CC_HIP(launch_gate_up_swiglu(W.w_gate, W.w_up, a, act, N, D, F, s));
    CC_HIP(launch_linear_residual(act, W.w_down, h, N, D, F, part, s));
  }
  CC_HIP(launch_rmsnorm(h, in->final_norm, a, N, D, p->rms_eps, s));
  return run_lmhead(p, a, in->w_lm, in->token_ids, scores, nullptr, at(ws, L.lm), s, 0,
                    in->w_lm_packed);
}

// The exact fast variant (Sec. 3.1, fast single-layer approximation): one layer of the
// full pass, entered with the stored activations H instead of the embedding stack, on
// the cache's last layer.
cc_status score_last_h(const cc_problem* p, const cc_inputs* in, float* scores, void* ws,
                       size_t ws_bytes, void* stream) {
  CC_TRY(check_kv(p, &in->kv, 1));
  const int N = n_tokens(p);
  if (N > 0 && (!in->h_last || !in->layers_h || !in->final_norm || !in->token_ids || !scores))
    return CC_ERR_ARG;
  if (N > 0) {
    if (!aligned16(in->h_last) || !lm_weight_ok(p, in->w_lm) || !aligned16(in->final_norm))
      return CC_ERR_ARG;
    const cc_layer_weights& W = in->layers_h[0];
    const void* ptrs[7] = {W.attn_norm, W.wq, W.wo, W.mlp_norm, W.w_gate, W.w_up, W.w_down};
    for (const void* q : ptrs)
      if (!q || !aligned16(q)) return CC_ERR_ARG;
  }
  CC_TRY(check_packed(p, in->w_lm_packed));
  const FullLayout L = full_layout(p);
  CC_TRY(check_ws(ws, ws_bytes, L.total));
  if (N == 0) return CC_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int D = p->hidden, F = p->ffn, HD = p->n_heads_q * p->head_dim;
  float2* rot = reinterpret_cast<float2*>(at(ws, L.rot));
  float* h = reinterpret_cast<float*>(at(ws, L.h));
  void* a = at(ws, L.a);
  void* q = at(ws, L.q);
  void* o = at(ws, L.o);
  void* act = at(ws, L.act);
  float* part = reinterpret_cast<float*>(at(ws, L.part));
  const cc_layer_weights& W = in->layers_h[0];
  CC_HIP(launch_rope_table(in->pos_ids, p->cu_seqlens_d, p->n_seqs, rot, N, p->head_dim,
                           double(p->rope_theta), s));
  CC_HIP(launch_embed(in->h_last, nullptr, h, N, D, s));   // widen H to the fp32 stream
  CC_HIP(launch_rmsnorm(h, W.attn_norm, a, N, D, p->rms_eps, s));
  CC_HIP(launch_qproj_rope(W.wq, a, q, rot, N, D, HD, part, s));
  CC_TRY(run_attention(p, q, &in->kv, in->kv.n_layers - 1, o, at(ws, L.attn), s));
  CC_HIP(launch_linear_residual(o, W.wo, h, N, D, HD, part, s));
  CC_HIP(launch_rmsnorm(h, W.mlp_norm, a, N, D, p->rms_eps, s));
  CC_HIP(launch_gate_up_swiglu(W.w_gate, W.w_up, a, act, N, D, F, s));
  CC_HIP(launch_linear_residual(act, W.w_down, h, N, D, F, part, s));
  CC_HIP(launch_rmsnorm(h, in->final_norm, a, N, D, p->rms_eps, s));
  return run_lmhead(p, a, in->w_lm, in->token_ids, scores, nullptr, at(ws, L.lm), s, 0,
                    in->w_lm_packed);
}

}  // namespace

extern "C" {

const char* cc_status_str(cc_status s) {
  switch (s) {
    case CC_OK: return "CC_OK";
    case CC_ERR_ARG: return "CC_ERR_ARG: invalid argument";
    case CC_ERR_SHAPE: return "CC_ERR_SHAPE: inconsistent sizes";
    case CC_ERR_DTYPE: return "CC_ERR_DTYPE: unsupported dtype for this call";
    case CC_ERR_WORKSPACE: return "CC_ERR_WORKSPACE: workspace too small";
    case CC_ERR_UNSUPPORTED: return "CC_ERR_UNSUPPORTED: no kernel for this shape";
    case CC_ERR_HIP: return "CC_ERR_HIP: HIP runtime error";
    case CC_ERR_SCRATCH: return "CC_ERR_SCRATCH: larger than the static scratch of the allocation-free entry point";
  }
  return "unknown cc_status";
}

const char* cc_version(void) { return "libcc gfx950 " __DATE__; }

cc_status cc_attention_workspace(const cc_problem* p, size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  *bytes = attention_ws_bytes(p);
  return CC_OK;
}

cc_status cc_attention_cc(const cc_problem* p, const void* q, const cc_kv* kv, int32_t layer,
                          void* o, void* ws, size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  CC_TRY(check_kv(p, kv, 1));
  if (layer < 0 || layer >= kv->n_layers) return CC_ERR_ARG;
  if (n_tokens(p) > 0 && (!q || !o)) return CC_ERR_ARG;
  if (p->dtype == CC_BF16 && (!aligned16(q) || !aligned16(o))) return CC_ERR_ARG;
  CC_TRY(check_ws(ws, ws_bytes, attention_ws_bytes(p)));
  return run_attention(p, q, kv, layer, o, ws, static_cast<hipStream_t>(stream));
}

cc_status cc_lmhead_workspace(const cc_problem* p, size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  *bytes = lmhead_ws_bytes(p);
  return CC_OK;
}

cc_status cc_lmhead_score(const cc_problem* p, const void* u, const void* w_lm,
                          const int32_t* token_ids, float* scores, float* lse, void* ws,
                          size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  if (n_tokens(p) > 0 && (!u || !w_lm || !token_ids || !scores)) return CC_ERR_ARG;
  if (p->dtype == CC_BF16 && (!aligned16(u) || !aligned16(w_lm))) return CC_ERR_ARG;
  if (p->lmhead_packed && n_tokens(p) > 0) return CC_ERR_ARG;   // cc_lmhead_score_packed
  CC_TRY(check_ws(ws, ws_bytes, lmhead_ws_bytes(p)));
  return run_lmhead(p, u, w_lm, token_ids, scores, lse, ws, static_cast<hipStream_t>(stream));
}

}  // extern "C"

// ------------------------------------------------------------------ allocation-free LM head
// The scratch of cc_lmhead_score_noalloc: a file-scope device array, one per GPU.  In host
// code its name is a host-side stand-in, not a device address, so it is never passed to a
// kernel or a copy; the device address comes from hipGetSymbolAddress, taken once per
// device with that device current and kept here.
namespace {
static __device__ __align__(256) unsigned char scratch[CC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The scratch's device address on the current device (looked up on its first use there).
cc_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return CC_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return CC_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return CC_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CC_OK;
}
}  // namespace

extern "C" {

cc_status cc_lmhead_score_noalloc(const cc_problem* p, const void* u, const void* w_lm,
                                  const int32_t* token_ids, float* scores, float* lse,
                                  void* stream) {
  CC_TRY(check_problem(p));
  if (p->lmhead_packed) return CC_ERR_ARG;
  if (n_tokens(p) > 0 && (!u || !w_lm || !token_ids || !scores)) return CC_ERR_ARG;
  if (p->dtype == CC_BF16 && (!aligned16(u) || !aligned16(w_lm))) return CC_ERR_ARG;
  const size_t need = lmhead_ws_bytes(p);
  if (need > CC_NOALLOC_SCRATCH_BYTES) return CC_ERR_SCRATCH;
  if (n_tokens(p) == 0) return CC_OK;
  void* ws = nullptr;
  CC_TRY(scratch_address(&ws));
  return run_lmhead(p, u, w_lm, token_ids, scores, lse, ws, static_cast<hipStream_t>(stream));
}

cc_status cc_lmhead_score_packed(const cc_problem* p, const void* u, const void* w_packed,
                                 const int32_t* token_ids, float* scores, float* lse, void* ws,
                                 size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  if (!p->lmhead_packed) return CC_ERR_ARG;
  if (n_tokens(p) > 0 && (!u || !token_ids || !scores)) return CC_ERR_ARG;
  if (!aligned16(u)) return CC_ERR_ARG;
  CC_TRY(check_packed(p, w_packed));
  CC_TRY(check_ws(ws, ws_bytes, lmhead_ws_bytes(p)));
  return run_lmhead(p, u, nullptr, token_ids, scores, lse, ws, static_cast<hipStream_t>(stream),
                    0, w_packed);
}

cc_status cc_pack_lmhead_bytes(int64_t rows, int32_t cols, size_t* bytes) {
  if (!bytes || rows < 0 || cols < 1 || cols % 32 != 0) return CC_ERR_ARG;
  *bytes = packed_rows_bytes(rows, cols);
  return CC_OK;
}

cc_status cc_pack_lmhead(const void* x, int64_t rows, int32_t cols, void* out,
                         size_t out_bytes, void* stream) {
  size_t need = 0;
  CC_TRY(cc_pack_lmhead_bytes(rows, cols, &need));
  if (rows == 0) return CC_OK;
  if (!x || !out || !aligned16(x) || !aligned16(out)) return CC_ERR_ARG;
  if (out_bytes < need) return CC_ERR_WORKSPACE;
  const char* xb = static_cast<const char*>(x);
  const char* ob = static_cast<const char*>(out);
  if (ob < xb + size_t(rows) * cols * 2 && xb < ob + need) return CC_ERR_ARG;   // overlap
  CC_HIP(launch_pack_rows(x, rows, cols, cols, out, static_cast<hipStream_t>(stream)));
  return CC_OK;
}

cc_status cc_linear(int32_t dtype, const void* x, const void* w, void* y, int32_t M, int32_t N,
                    int32_t K, void* stream) {
  if (dtype != CC_F32 && dtype != CC_BF16) return CC_ERR_DTYPE;
  if (M < 0 || N < 0 || K < 1) return CC_ERR_SHAPE;
  if (M > 0 && N > 0 && (!x || !w || !y)) return CC_ERR_ARG;
  if (dtype == CC_BF16) {
    if (K % 64 != 0) return CC_ERR_UNSUPPORTED;
    if (!aligned16(x) || !aligned16(w)) return CC_ERR_ARG;
  }
  CC_HIP(launch_linear(dtype, x, w, y, M, N, K, static_cast<hipStream_t>(stream)));
  return CC_OK;
}

cc_status cc_score_workspace(const cc_problem* p, size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  const bool last = p->mode == CC_MODE_LAST_LAYER || p->mode == CC_MODE_LAST_LAYER_FUSED;
  *bytes = last ? score_layout(p).total : full_layout(p).total;
  return CC_OK;
}

cc_status cc_score(const cc_problem* p, const cc_inputs* in, float* scores, void* ws,
                   size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  if (!in) return CC_ERR_ARG;
  if (p->mode == CC_MODE_FULL) return score_full(p, in, scores, ws, ws_bytes, stream);
  if (p->mode == CC_MODE_LAST_LAYER_H) return score_last_h(p, in, scores, ws, ws_bytes, stream);
  CC_TRY(check_kv(p, &in->kv, 1));
  const int N = n_tokens(p);
  const bool fused = p->mode == CC_MODE_LAST_LAYER_FUSED;
  if (N > 0 && (!in->q || (!fused && !in->w_o) || !in->token_ids || !scores)) return CC_ERR_ARG;
  if (N > 0 && !p->lmhead_packed && !in->w_lm) return CC_ERR_ARG;
  if (p->dtype == CC_BF16 &&
      (!aligned16(in->q) || (!fused && !aligned16(in->w_o)) || !lm_weight_ok(p, in->w_lm)))
    return CC_ERR_ARG;
  CC_TRY(check_packed(p, in->w_lm_packed));
  const ScoreLayout L = score_layout(p);
  CC_TRY(check_ws(ws, ws_bytes, L.total));
  if (N == 0) return CC_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* o = at(ws, L.o);
  void* u = at(ws, L.u);
  CC_TRY(run_attention(p, in->q, &in->kv, in->kv.n_layers - 1, o, at(ws, L.attn), s));
  const int qdim = p->n_heads_q * p->head_dim;
  if (fused)   // z = (W_lm W_o) y straight from the attention rows
    return run_lmhead(p, o, in->w_lm, in->token_ids, scores, nullptr, at(ws, L.lm), s, qdim,
                      in->w_lm_packed);
  CC_HIP(launch_linear(p->dtype, o, in->w_o, u, N, p->hidden, qdim, s));
  return run_lmhead(p, u, in->w_lm, in->token_ids, scores, nullptr, at(ws, L.lm), s, 0,
                    in->w_lm_packed);
}

// ------------------------------------------------------------------ fused LM-head weight

cc_status cc_fuse_wo_lmhead_workspace(int32_t dtype, int32_t hidden, int32_t qdim,
                                      size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  if (dtype != CC_F32 && dtype != CC_BF16) return CC_ERR_DTYPE;
  if (hidden < 1 || qdim < 1) return CC_ERR_SHAPE;
  *bytes = align_up(size_t(hidden) * qdim * esize(dtype));
  return CC_OK;
}

cc_status cc_fuse_wo_lmhead(int32_t dtype, const void* w_lm, const void* w_o, void* out,
                            int32_t vocab, int32_t hidden, int32_t qdim, void* ws,
                            size_t ws_bytes, void* stream) {
  if (dtype != CC_F32 && dtype != CC_BF16) return CC_ERR_DTYPE;
  if (vocab < 1 || hidden < 1 || qdim < 1) return CC_ERR_SHAPE;
  if (!w_lm || !w_o || !out) return CC_ERR_ARG;
  if (dtype == CC_BF16) {
    if (hidden % 64 != 0) return CC_ERR_UNSUPPORTED;
    if (!aligned16(w_lm) || !aligned16(w_o) || !aligned16(out)) return CC_ERR_ARG;
  }
  CC_TRY(check_ws(ws, ws_bytes, align_up(size_t(hidden) * qdim * esize(dtype))));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // W_o [hidden][qdim] -> W_o^T [qdim][hidden] (K-contiguous), then out = W_lm (W_o^T)^T
  CC_HIP(launch_transpose(dtype, w_o, ws, hidden, qdim, s));
  CC_HIP(launch_linear(dtype, w_lm, ws, out, vocab, qdim, hidden, s));
  return CC_OK;
}

// ------------------------------------------------------------------ FP8 LM head

cc_status cc_quantize_fp8_workspace(int64_t rows, size_t* bytes) {
  if (!bytes || rows < 0) return CC_ERR_ARG;
  *bytes = align_up(size_t(rows + 1) * sizeof(float));
  return CC_OK;
}

cc_status cc_quantize_fp8(int32_t dtype, const void* x, int64_t rows, int32_t cols,
                          int32_t per_row, uint8_t* codes, float* scale, void* ws,
                          size_t ws_bytes, void* stream) {
  if (dtype != CC_F32 && dtype != CC_BF16) return CC_ERR_DTYPE;
  if (rows < 0 || rows > INT32_MAX || cols < 4 || cols % 4 != 0) return CC_ERR_SHAPE;
  if (per_row != 0 && per_row != 1) return CC_ERR_ARG;
  if (rows == 0) return CC_OK;
  if (!x || !codes || !scale) return CC_ERR_ARG;
  if ((reinterpret_cast<uintptr_t>(codes) & 3u) != 0) return CC_ERR_ARG;
  if ((reinterpret_cast<uintptr_t>(x) & uintptr_t(4 * esize(dtype) - 1)) != 0) return CC_ERR_ARG;
  CC_TRY(check_ws(ws, ws_bytes, align_up(size_t(rows + 1) * sizeof(float))));
  CC_HIP(launch_quantize_e4m3(dtype, x, rows, cols, per_row, codes, scale,
                              static_cast<float*>(ws), static_cast<hipStream_t>(stream)));
  return CC_OK;
}

namespace {
struct Fp8Layout {
  size_t uq, su, amax, partial, target, total;
};
Fp8Layout fp8_layout(const cc_problem* p) {
  Fp8Layout L;
  const size_t N = n_tokens(p), D = p->hidden;
  const size_t n_vt = (p->vocab + 255) / 256;
  size_t off = 0;
  L.uq = off;
  off += align_up(N * D);
  L.su = off;
  off += align_up(N * sizeof(float));
  L.amax = off;
  off += align_up((N + 1) * sizeof(float));
  L.partial = off;
  off += align_up(n_vt * N * sizeof(float2));
  L.target = off;
  off += align_up(N * sizeof(float));
  L.total = off;
  return L;
}
}  // namespace

cc_status cc_lmhead_fp8_workspace(const cc_problem* p, size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  *bytes = fp8_layout(p).total;
  return CC_OK;
}

cc_status cc_lmhead_score_fp8(const cc_problem* p, const void* u, const uint8_t* w_codes,
                              const float* w_scale, const int32_t* token_ids, float* scores,
                              float* lse, void* ws, size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  if (p->hidden % 128 != 0) return CC_ERR_UNSUPPORTED;
  const int N = n_tokens(p);
  if (N > 0 && (!u || !w_codes || !w_scale || !token_ids || !scores)) return CC_ERR_ARG;
  if (N > 0 && !aligned16(w_codes)) return CC_ERR_ARG;
  if (N > 0 && (reinterpret_cast<uintptr_t>(u) & uintptr_t(4 * esize(p->dtype) - 1)) != 0)
    return CC_ERR_ARG;
  const Fp8Layout L = fp8_layout(p);
  CC_TRY(check_ws(ws, ws_bytes, L.total));
  if (N == 0) return CC_OK;
  LmHeadFp8Launch a;
  a.dtype = p->dtype;
  a.u = u;
  a.wq = w_codes;
  a.sw = w_scale;
  a.ids = token_ids;
  a.scores = scores;
  a.lse = lse;
  a.uq = reinterpret_cast<uint8_t*>(at(ws, L.uq));
  a.su = reinterpret_cast<float*>(at(ws, L.su));
  a.amax_ws = reinterpret_cast<float*>(at(ws, L.amax));
  a.partial = reinterpret_cast<float2*>(at(ws, L.partial));
  a.target = reinterpret_cast<float*>(at(ws, L.target));
  a.cu_d = p->cu_seqlens_d;
  a.n_seqs = p->n_seqs;
  a.N = N;
  a.D = p->hidden;
  a.V = p->vocab;
  a.n_frozen = p->n_frozen;
  CC_HIP(launch_lmhead_fp8(a, static_cast<hipStream_t>(stream)));
  return CC_OK;
}

// ------------------------------------------------------------------ selection

cc_status cc_select_workspace(int32_t n_segs, size_t* bytes) {
  if (!bytes || n_segs < 0) return CC_ERR_ARG;
  *bytes = align_up(size_t(n_segs) * sizeof(SelSeg));
  return CC_OK;
}

cc_status cc_select_keep(const float* scores, int32_t n_segs, const int64_t* seg_start_h,
                         const int32_t* seg_len_h, const int32_t* k_h, int32_t* keep_idx,
                         void* ws, size_t ws_bytes, void* stream) {
  if (n_segs < 0) return CC_ERR_ARG;
  if (n_segs == 0) return CC_OK;
  if (!seg_start_h || !seg_len_h || !k_h) return CC_ERR_ARG;
  std::vector<SelSeg> segs(n_segs);
  int64_t out = 0;
  int mx = 0;
  bool any_len = false;
  for (int i = 0; i < n_segs; ++i) {
    if (seg_len_h[i] < 0 || seg_start_h[i] < 0) return CC_ERR_SHAPE;
    if (k_h[i] < 0 || k_h[i] > seg_len_h[i]) return CC_ERR_SHAPE;
    segs[i].start = seg_start_h[i];
    segs[i].len = seg_len_h[i];
    segs[i].k = k_h[i];
    segs[i].out = out;
    out += k_h[i];
    mx = std::max(mx, seg_len_h[i]);
    any_len = any_len || (k_h[i] > 0);
  }
  if (any_len && (!scores || !keep_idx)) return CC_ERR_ARG;
  CC_TRY(check_ws(ws, ws_bytes, align_up(size_t(n_segs) * sizeof(SelSeg))));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // a few descriptors travel in the kernel arguments, regular layouts as a formula; others
  // are copied into the workspace
  if (n_segs > SEL_INLINE && !select_regular(segs.data(), n_segs))
    CC_HIP(hipMemcpyAsync(ws, segs.data(), segs.size() * sizeof(SelSeg), hipMemcpyHostToDevice, s));
  CC_HIP(launch_select(scores, segs.data(), static_cast<const SelSeg*>(ws), n_segs, mx, keep_idx, s));
  return CC_OK;
}

// ------------------------------------------------------------------ compaction

namespace {
struct CompactPlan {
  std::vector<CompactList> lists;
  std::vector<CompactPlane> planes;
  std::vector<int32_t> seq_list;
  int max_k = 0;
  size_t off_lists = 0, off_planes = 0, off_seq = 0, total = 0;
};

size_t compact_ws_bytes_for(const cc_problem* p, int per_head, int n_layers) {
  const size_t n_lists = size_t(p->n_seqs) * (per_head ? p->n_heads_kv : 1);
  const size_t n_planes = size_t(p->n_seqs) * n_layers * p->n_heads_kv;
  return align_up(n_lists * sizeof(CompactList)) + align_up(n_planes * sizeof(CompactPlane)) +
         align_up(size_t(p->n_seqs) * sizeof(int32_t));
}
}  // namespace

cc_status cc_compact_workspace(const cc_problem* p, int32_t cache_layers, int32_t per_head,
                               size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  if (per_head != 0 && per_head != 1) return CC_ERR_ARG;
  if (cache_layers < 1) return CC_ERR_ARG;
  *bytes = compact_ws_bytes_for(p, per_head, cache_layers);
  return CC_OK;
}

cc_status cc_compact_kv(const cc_problem* p, const cc_kv* kv, const int32_t* keep_idx,
                        const int32_t* k_h, int32_t per_head, int32_t* token_ids,
                        int32_t* pos_ids, const cc_kv* out, void* ws, size_t ws_bytes,
                        void* stream) {
  CC_TRY(check_problem(p));
  CC_TRY(check_kv(p, kv, 1));
  if (per_head != 0 && per_head != 1) return CC_ERR_ARG;
  if (!k_h) return CC_ERR_ARG;
  if (out) {
    CC_TRY(check_kv(p, out, kv->n_layers));
    if (out->layout != kv->layout) return CC_ERR_ARG;
  }
  const int es = esize(p->dtype);
  const int row_bytes = p->head_dim * es;
  if (row_bytes % 16 != 0 || !is_pow2(row_bytes / 16) || row_bytes / 16 > 256)
    return CC_ERR_UNSUPPORTED;
  const int hkv = p->n_heads_kv;
  const int n_lists = p->n_seqs * (per_head ? hkv : 1);
  CompactPlan plan;
  plan.lists.resize(n_lists);
  int64_t off = 0;
  for (int b = 0; b < p->n_seqs; ++b) {
    const int n = p->cu_seqlens_h[b + 1] - p->cu_seqlens_h[b];
    for (int h = 0; h < (per_head ? hkv : 1); ++h) {
      const int li = per_head ? b * hkv + h : b;
      const int k = k_h[li];
      if (k < 0 || k > n) return CC_ERR_SHAPE;
      plan.lists[li].keep_off = off;
      plan.lists[li].tok0 = 0;
      plan.lists[li].k = k;
      plan.lists[li].pad = 0;
      off += k;
      plan.max_k = std::max(plan.max_k, k);
    }
  }
  if (off > 0 && !keep_idx) return CC_ERR_ARG;
  plan.seq_list.resize(p->n_seqs);
  for (int b = 0; b < p->n_seqs; ++b) plan.seq_list[b] = per_head ? b * hkv : b;
  const int L = kv->n_layers;
  for (int b = 0; b < p->n_seqs; ++b)
    for (int l = 0; l < L; ++l)
      for (int h = 0; h < hkv; ++h) {
        const int li = per_head ? b * hkv + h : b;
        if (plan.lists[li].k == 0) continue;
        plan.planes.push_back(CompactPlane{b, l, h, li});
      }
  std::stable_sort(plan.planes.begin(), plan.planes.end(),
                   [&](const CompactPlane& a, const CompactPlane& c) {
                     return plan.lists[a.list].k > plan.lists[c.list].k;
                   });
  plan.off_lists = 0;
  plan.off_planes = align_up(plan.lists.size() * sizeof(CompactList));
  plan.off_seq = plan.off_planes + align_up(size_t(p->n_seqs) * L * hkv * sizeof(CompactPlane));
  plan.total = plan.off_seq + align_up(size_t(p->n_seqs) * sizeof(int32_t));
  if (plan.total != compact_ws_bytes_for(p, per_head, L)) return CC_ERR_ARG;
  CC_TRY(check_ws(ws, ws_bytes, plan.total));
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the three tables go up as one host image of the workspace prefix: one copy, not three
  // (each copy from pageable memory is a separate transfer on the stream)
  std::vector<char> img(plan.off_seq + plan.seq_list.size() * sizeof(int32_t));
  std::memcpy(img.data() + plan.off_lists, plan.lists.data(), plan.lists.size() * sizeof(CompactList));
  if (!plan.planes.empty())
    std::memcpy(img.data() + plan.off_planes, plan.planes.data(),
                plan.planes.size() * sizeof(CompactPlane));
  std::memcpy(img.data() + plan.off_seq, plan.seq_list.data(), plan.seq_list.size() * sizeof(int32_t));
  CC_HIP(hipMemcpyAsync(ws, img.data(), img.size(), hipMemcpyHostToDevice, s));
  CompactLaunch c;
  c.n_tensors = 2;
  const cc_kv* dst = out ? out : kv;
  c.src[0] = make_view(kv, kv->k, es);
  c.src[1] = make_view(kv, kv->v, es);
  c.dst[0] = make_view(dst, dst->k, es);
  c.dst[1] = make_view(dst, dst->v, es);
  c.paged = kv->layout == CC_KV_PAGED;
  c.row_bytes = row_bytes;
  c.keep = keep_idx;
  c.lists_d = reinterpret_cast<const CompactList*>(at(ws, plan.off_lists));
  c.planes_d = reinterpret_cast<const CompactPlane*>(at(ws, plan.off_planes));
  c.n_planes = int(plan.planes.size());
  c.max_k = plan.max_k;
  c.in_place = out == nullptr;
  c.ids[0] = token_ids;
  c.ids[1] = pos_ids;
  c.cu_d = p->cu_seqlens_d;
  c.seq_list_d = reinterpret_cast<const int32_t*>(at(ws, plan.off_seq));
  c.n_seqs = p->n_seqs;
  CC_HIP(launch_compact(c, s));
  return CC_OK;
}

// Token-major per-entry rows (e.g. the stored activations H) follow the keep lists of
// the cache.  The rows are cut into column slabs of up to 256 bytes; each (sequence, slab)
// is one plane of the compaction kernels, addressed through a flat view whose planes
// start at the sequence's first row.
namespace {
int rows_slab_bytes(int row_bytes) {
  int slab = 256;
  while (slab > 16 && row_bytes % slab != 0) slab >>= 1;
  return slab;
}
size_t rows_ws_bytes(const cc_problem* p, int row_bytes) {
  const size_t n_slabs = size_t(row_bytes / rows_slab_bytes(row_bytes));
  return align_up(size_t(p->n_seqs) * sizeof(CompactList)) +
         align_up(size_t(p->n_seqs) * n_slabs * sizeof(CompactPlane));
}
}  // namespace

cc_status cc_compact_rows_workspace(const cc_problem* p, int32_t row_bytes, int32_t per_head,
                                    size_t* bytes) {
  if (!bytes) return CC_ERR_ARG;
  CC_TRY(check_problem(p));
  if (per_head != 0 && per_head != 1) return CC_ERR_ARG;
  if (row_bytes < 16 || row_bytes % 16 != 0) return CC_ERR_UNSUPPORTED;
  *bytes = rows_ws_bytes(p, row_bytes);
  return CC_OK;
}

cc_status cc_compact_rows(const cc_problem* p, void* rows, int32_t row_bytes,
                          const int32_t* keep_idx, const int32_t* k_h, int32_t per_head,
                          void* out_rows, void* ws, size_t ws_bytes, void* stream) {
  CC_TRY(check_problem(p));
  if (per_head != 0 && per_head != 1) return CC_ERR_ARG;
  if (row_bytes < 16 || row_bytes % 16 != 0) return CC_ERR_UNSUPPORTED;
  if (!k_h) return CC_ERR_ARG;
  const int hkv = p->n_heads_kv;
  const int slab = rows_slab_bytes(row_bytes), n_slabs = row_bytes / slab;
  std::vector<CompactList> lists(p->n_seqs);
  std::vector<CompactPlane> planes;
  int64_t off = 0;
  int max_k = 0;
  for (int b = 0; b < p->n_seqs; ++b) {
    const int n = p->cu_seqlens_h[b + 1] - p->cu_seqlens_h[b];
    for (int h = 0; h < (per_head ? hkv : 1); ++h) {
      const int li = per_head ? b * hkv + h : b;
      if (k_h[li] < 0 || k_h[li] > n) return CC_ERR_SHAPE;
      if (h == 0) {   // the sequence's first list
        lists[b].keep_off = off;
        lists[b].tok0 = p->cu_seqlens_h[b];
        lists[b].k = k_h[li];
        lists[b].pad = 0;
        max_k = std::max(max_k, k_h[li]);
      }
      off += k_h[li];
    }
  }
  if (off > 0 && (!keep_idx || !rows)) return CC_ERR_ARG;
  if ((rows && !aligned16(rows)) || (out_rows && !aligned16(out_rows))) return CC_ERR_ARG;
  for (int b = 0; b < p->n_seqs; ++b)
    if (lists[b].k > 0)
      for (int h = 0; h < n_slabs; ++h) planes.push_back(CompactPlane{b, 0, h, b});
  const size_t off_planes = align_up(size_t(p->n_seqs) * sizeof(CompactList));
  CC_TRY(check_ws(ws, ws_bytes, rows_ws_bytes(p, row_bytes)));
  if (planes.empty()) return CC_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // both tables as one host image of the workspace prefix (one copy)
  std::vector<char> img(off_planes + planes.size() * sizeof(CompactPlane));
  std::memcpy(img.data(), lists.data(), lists.size() * sizeof(CompactList));
  std::memcpy(img.data() + off_planes, planes.data(), planes.size() * sizeof(CompactPlane));
  CC_HIP(hipMemcpyAsync(ws, img.data(), img.size(), hipMemcpyHostToDevice, s));
  auto view = [&](void* base) {
    KvView v{};
    v.base = base;
    v.head_stride = slab;      // bytes: column slab h
    v.tok_stride = row_bytes;  // bytes: one entry
    return v;
  };
  CompactLaunch c;
  c.n_tensors = 1;
  c.src[0] = c.src[1] = view(rows);
  c.dst[0] = c.dst[1] = view(out_rows ? out_rows : rows);
  c.paged = false;
  c.row_bytes = slab;
  c.keep = keep_idx;
  c.lists_d = static_cast<const CompactList*>(ws);
  c.planes_d = reinterpret_cast<const CompactPlane*>(at(ws, off_planes));
  c.n_planes = int(planes.size());
  c.max_k = max_k;
  c.in_place = out_rows == nullptr;
  c.ids[0] = c.ids[1] = nullptr;
  c.cu_d = p->cu_seqlens_d;
  c.seq_list_d = nullptr;
  c.n_seqs = 0;
  CC_HIP(launch_compact(c, s));
  return CC_OK;
}

}  // extern "C"
