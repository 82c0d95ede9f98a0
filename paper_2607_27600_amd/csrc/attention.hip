// Counter-causal attention (Eq. (2) under the mask of Sec. 3.1): every cached entry i
// attends only to later entries j > i of its own sequence, reusing the stored keys and
// values.  Output o[i][h] = sum_j softmax_j(scale * q[i][h] . k[j][c]) v[j][c], c = h/g.
//
// bf16 path (head_dim 128): flash-style, one workgroup of 4 waves per (sequence, KV head,
// block of 128 "rows"), where a row is one (position, query head of the GQA group) pair,
// so the g query heads that share a KV head share every K/V tile staged in LDS.
//   S^T = K Q^T and O^T = V^T P^T on 32x32x16 bf16 MFMA.  Computing the transposed
//   products leaves each lane owning one query row (column of the MFMA output), so the
//   online-softmax statistics and rescaling stay in registers of that lane; the P tile
//   feeds the second MFMA straight from registers.
//   Key tiles entirely at or before the block's first row are never visited (they are
//   masked for every row), so the work per block shrinks towards the end of the
//   sequence; only tiles that straddle the diagonal or the sequence end are masked.
//   K tiles are stored row-major in LDS, V tiles transposed with the key order permuted
//   to match the MFMA k-slots of the P operand; both are double buffered with one
//   barrier per tile.
// fp32 path: one thread per row, K/V tiles staged in LDS, exact fp32 online softmax.
#include <type_traits>

#include "cc_internal.h"

namespace cc {
namespace {

#define SCHED_VALU 0x002
#define SCHED_MFMA 0x008
#define SCHED_DS_READ 0x100
#define SCHED_TRANS 0x400

constexpr int BN = 64;            // keys per tile
constexpr int HD = 128;           // head dim of the MFMA path
constexpr int ROWS_W = 32;        // rows per wave
constexpr int NWAVES = 4;
constexpr int ROWS = ROWS_W * NWAVES;
constexpr int KS = HD + 8;        // LDS row stride of K (elements): 272 B
constexpr int VS = BN + 8;        // LDS row stride of V^T (elements): 144 B
constexpr int K_TILE = BN * KS;
constexpr int V_TILE = HD * VS;
constexpr float kRescale = 8.f;   // log2 headroom before the softmax reference max moves

struct AttnArgs {
  const u16* q;
  u16* o;
  const int32_t* cu;
  const int4* work;
  KvView k, v;
  int layer;
  int hq, g;
  float c2;        // scale * log2(e)
  int inclusive;
};

__device__ __forceinline__ uint4 ld16(const u16* p) { return *reinterpret_cast<const uint4*>(p); }

template <bool PAGED>
__global__ __launch_bounds__(256, 2) void attn_cc_bf16(AttnArgs a) {
  // K tiles run one tile ahead of V tiles: while the softmax of tile t runs on the VALU, the
  // MFMAs of S for tile t+1 are already issued, so each wave overlaps its own softmax with
  // matrix work.  Two K buffers (tiles t+1, t+2) and two V buffers (tiles t, t+1).
  __shared__ __attribute__((aligned(16))) u16 kl[2][K_TILE];
  __shared__ __attribute__((aligned(16))) u16 vl[2][V_TILE];

  const int4 w = a.work[blockIdx.x];
  const int b = w.x, kvh = w.y, rb = w.z;
  const int seq0 = a.cu[b];
  const int n = a.cu[b + 1] - seq0;
  const int g = a.g;
  const int nrows = n * g;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int hi = lane >> 5, col = lane & 31;

  const int row = rb * ROWS + wave * ROWS_W + col;
  const bool valid = row < nrows;
  const int pos = valid ? row / g : n;
  const int hq = kvh * g + (valid ? row % g : 0);

  // This lane's query row as the B operand of S^T = K Q^T: 8 k-steps of 16 dims,
  // lane half `hi` holds dims ks*16 + hi*8 .. +7.
  bf16x8 qf[8];
  {
    const u16* qp = a.q + (int64_t(seq0 + (valid ? pos : 0)) * a.hq + hq) * HD + hi * 8;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 v = valid ? ld16(qp + ks * 16) : make_uint4(0, 0, 0, 0);
      qf[ks] = as_bf16x8(v);
    }
  }

  const int row0 = rb * ROWS;
  const int pos_lo = row0 / g;
  const int wg_last = min(row0 + ROWS, nrows) - 1;
  const int pos_hi_wg = row0 + ROWS > nrows ? n : wg_last / g;   // partial blocks mask always
  const int first_key = pos_lo + (a.inclusive ? 0 : 1);
  const int tb = first_key / BN;
  const int te = (n + BN - 1) / BN;
  if (tb >= te) {
    // no key reachable from any row of the block: every output row is 0
    if (valid) {
      u16* op = a.o + (int64_t(seq0 + pos) * a.hq + hq) * HD + hi * 4;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          *reinterpret_cast<uint2*>(op + db * 32 + jj * 8) = make_uint2(0, 0);
    }
    return;
  }
  // tiles [tb, tm0) and [tm1, te) need the mask; [tm0, tm1) see every key of every row
  const int tm0 = min(te, max(tb, (pos_hi_wg + 1 + BN - 1) / BN));
  const int tm1 = (n % BN == 0) ? te : te - 1;

  const u16* kbase = reinterpret_cast<const u16*>(a.k.base);
  const u16* vbase = reinterpret_cast<const u16*>(a.v.base);

  // global -> register staging
  // K: thread owns 16-byte column chunk kc of rows kr0 + 16*i.
  const int kc = tid & 15, kr0 = tid >> 4;
  // V: thread owns keys 4*vg .. 4*vg+3, dims 8*vd .. 8*vd+7.
  const int vg = tid & 15, vd = tid >> 4;
  uint4 kreg[4], vreg[4];

  // Row addressing.  Contiguous caches: this thread's rows of tile 0 are fixed pointers
  // and a tile is a uniform (scalar) offset, so full tiles cost one add per row; only the
  // last, partial tile clamps rows to n-1.  Paged caches: one block-table lookup per row.
  const u16* kp[4];
  const u16* vp[4];
  if constexpr (!PAGED) {
    const u16* kplane = kbase + kv_off<false>(a.k, b, a.layer, kvh, 0);
    const u16* vplane = vbase + kv_off<false>(a.v, b, a.layer, kvh, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      kp[i] = kplane + int64_t(kr0 + 16 * i) * a.k.tok_stride + kc * 8;
      vp[i] = vplane + int64_t(4 * vg + i) * a.v.tok_stride + vd * 8;
    }
  }
  auto load_k = [&](int t) {
    const int key0 = t * BN;   // rows past n are clamped to n-1 and masked
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        kreg[i] = ld16(kbase + kv_off<true>(a.k, b, a.layer, kvh, min(key0 + kr0 + 16 * i, n - 1)) +
                       kc * 8);
    } else {
      if (key0 + BN <= n) {
        const int64_t off = int64_t(key0) * a.k.tok_stride;
#pragma unroll
        for (int i = 0; i < 4; ++i) kreg[i] = ld16(kp[i] + off);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = min(key0 + kr0 + 16 * i, n - 1);
          kreg[i] = ld16(kp[i] + (int64_t(key - kr0 - 16 * i) * a.k.tok_stride));
        }
      }
    }
  };
  auto load_v = [&](int t) {
    const int key0 = t * BN;
    if constexpr (PAGED) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = key0 + 4 * vg + i;
        // value rows past n get zero (their weights are 0, but garbage could be NaN)
        vreg[i] = key < n ? ld16(vbase + kv_off<true>(a.v, b, a.layer, kvh, key) + vd * 8)
                          : make_uint4(0, 0, 0, 0);
      }
    } else {
      const int64_t off = int64_t(key0) * a.v.tok_stride;
      if (key0 + BN <= n) {
#pragma unroll
        for (int i = 0; i < 4; ++i) vreg[i] = ld16(vp[i] + off);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          vreg[i] = key0 + 4 * vg + i < n ? ld16(vp[i] + off) : make_uint4(0, 0, 0, 0);
      }
    }
  };
  // position of key 4*vg within the permuted V^T row (see the PV operand layout below)
  const int vpos = (vg >> 2) * 16 + (vg & 1) * 8 + ((vg >> 1) & 1) * 4;
  auto store_k = [&](u16* Kl) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<uint4*>(Kl + (kr0 + 16 * i) * KS + kc * 8) = kreg[i];
  };
  auto store_v = [&](u16* Vl) {
    const uint32_t* r0 = reinterpret_cast<const uint32_t*>(&vreg[0]);
    const uint32_t* r1 = reinterpret_cast<const uint32_t*>(&vreg[1]);
    const uint32_t* r2 = reinterpret_cast<const uint32_t*>(&vreg[2]);
    const uint32_t* r3 = reinterpret_cast<const uint32_t*>(&vreg[3]);
#pragma unroll
    for (int wd = 0; wd < 4; ++wd) {
      // dims 8*vd + 2*wd (low halves) and 8*vd + 2*wd + 1 (high halves)
      uint2 lo, hi2;
      lo.x = (r0[wd] & 0xffffu) | (r1[wd] << 16);
      lo.y = (r2[wd] & 0xffffu) | (r3[wd] << 16);
      hi2.x = (r0[wd] >> 16) | (r1[wd] & 0xffff0000u);
      hi2.y = (r2[wd] >> 16) | (r3[wd] & 0xffff0000u);
      const int d0 = vd * 8 + 2 * wd;
      *reinterpret_cast<uint2*>(Vl + d0 * VS + vpos) = lo;
      *reinterpret_cast<uint2*>(Vl + (d0 + 1) * VS + vpos) = hi2;
    }
  };

  // S^T[key][row] for the 64 keys of a tile: two 32-key blocks; 16 MFMAs, MFMA j uses
  // key block j%2 and dims 16*(j/2) ..
  auto kfrag = [&](const u16* Kl, int j) {
    return as_bf16x8(ld16(Kl + ((j & 1) * 32 + col) * KS + (j >> 1) * 16 + hi * 8));
  };
  auto vfrag = [&](const u16* Vl, int j) {   // PV MFMA j: k-step j/4, d block j%4
    return as_bf16x8(ld16(Vl + ((j & 3) * 32 + col) * VS + (j >> 2) * 16 + hi * 8));
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 acc[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) acc[db] = f32x16{};

  // prologue: K(tb), V(tb) and K(tb+1) in LDS, S(tb) in registers
  load_k(tb);
  load_v(tb);
  store_k(kl[0]);
  store_v(vl[0]);
  load_k(min(tb + 1, te - 1));
  store_k(kl[1]);
  __syncthreads();
  f32x16 s_cur[2], s_nxt[2];
  s_cur[0] = f32x16{};
  s_cur[1] = f32x16{};
#pragma unroll
  for (int j = 0; j < 16; ++j) s_cur[j & 1] = mfma32(kfrag(kl[0], j), qf[j >> 1], s_cur[j & 1]);

  // One tile.  S(t) is in s_cur; K(t+1) sits in kl[(t+1-tb)&1] and V(t) in vl[(t-tb)&1]; the
  // loads of K(t+2), V(t+1) refill the buffers freed by K(t), V(t-1).  The step is written
  // in the order it should issue (sched_barrier fences keep the compiler from regrouping):
  // the 16 MFMAs of S(t+1) are spread over the exponentials of this tile's softmax, and the
  // 16 MFMAs of P V over the LDS stores of the next tiles.  Past the last tile, loads and
  // S are clamped to the last tile and land in buffers nobody reads.
  auto step = [&](int t, auto mask_tag) {
    constexpr bool kMask = decltype(mask_tag)::value;
    const int i = t - tb;
    const u16* Kn = kl[(i + 1) & 1];
    const u16* Vc = vl[i & 1];
    load_k(min(t + 2, te - 1));
    load_v(min(t + 1, te - 1));
    bf16x8 kf[4];
    kf[0] = kfrag(Kn, 0);
    kf[1] = kfrag(Kn, 1);
    kf[2] = kfrag(Kn, 2);
    if (kMask) {
      const int key0 = t * BN;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          const bool ok = key < n && (a.inclusive ? key >= pos : key > pos);
          s_cur[mb][e] = ok ? s_cur[mb][e] : -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s_cur[mb][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    // Lazy rescaling: the reference max only moves when the row max grows by more than
    // 2^8 in probability units (or on the first non-empty tile).  Numerator and
    // denominator always share the reference, so the result is unchanged; p stays <= 256.
    const bool up = mx > m_run + kRescale / a.c2;
    const float corr = up ? fast_exp2((m_run - mx) * a.c2) : 1.f;   // 0 when m_run = -inf
    m_run = up ? mx : m_run;
    const float mc = (m_run == -INFINITY ? 0.f : m_run) * a.c2;
    s_nxt[0] = f32x16{};
    s_nxt[1] = f32x16{};
    float lsum = 0.f;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j + 3 < 16) kf[(j + 3) & 3] = kfrag(Kn, j + 3);
      s_nxt[j & 1] = mfma32(kf[j & 3], qf[j >> 1], s_nxt[j & 1]);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int f = 2 * j + u, mb = f >> 4, e = f & 15;
        const float p = fast_exp2(fmaf(s_cur[mb][e], a.c2, -mc));
        // pin the exponential here, between the MFMAs, instead of next to its later uses
        asm volatile("" ::"v"(p));
        s_cur[mb][e] = p;
        lsum += p;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    l_run = l_run * corr + lsum;
    // P^T operand: k-step kk covers keys 16*kk .. 16*kk+15; lane half hi holds keys
    // {4hi..4hi+3, 8+4hi..8+4hi+3} of that step, i.e. S^T entries 8*(kk%2)..+7 of block kk/2
    bf16x8 pf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kk][e] = (__bf16)s_cur[kk >> 1][(kk & 1) * 8 + e];
    if (__any(corr != 1.f)) {
#pragma unroll
      for (int db = 0; db < 4; ++db) acc[db] *= corr;
    }
    bf16x8 vf[4];
    vf[0] = vfrag(Vc, 0);
    vf[1] = vfrag(Vc, 1);
    vf[2] = vfrag(Vc, 2);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (j + 3 < 16) vf[(j + 3) & 3] = vfrag(Vc, j + 3);
      acc[j & 3] = mfma32(vf[j & 3], pf[j >> 2], acc[j & 3]);
      if (j == 7) store_k(kl[i & 1]);
      if (j == 11) store_v(vl[(i + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    s_cur[0] = s_nxt[0];
    s_cur[1] = s_nxt[1];
  };
  int t = tb;
  for (; t < tm0; ++t) step(t, std::true_type{});
  for (; t < tm1; ++t) step(t, std::false_type{});
  for (; t < te; ++t) step(t, std::true_type{});

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (valid) {
    u16* op = a.o + (int64_t(seq0 + pos) * a.hq + hq) * HD + hi * 4;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)(acc[db][jj * 4 + e] * inv);
        *reinterpret_cast<bf16x4*>(op + db * 32 + jj * 8) = o;
      }
  }
}

// ------------------------------------------------------------------ fp32 path

constexpr int F_ROWS = 128;   // rows (one per thread) per workgroup
constexpr int F_BN = 32;      // keys per LDS tile

struct AttnArgsF {
  const float* q;
  float* o;
  const int32_t* cu;
  const int4* work;
  KvView k, v;
  int layer;
  int hq, g;
  float scale;
  int inclusive;
};

template <int D, bool PAGED>
__global__ __launch_bounds__(F_ROWS) void attn_cc_f32(AttnArgsF a) {
  __shared__ float Ks[F_BN][D + 1];
  __shared__ float Vs[F_BN][D + 1];
  const int4 w = a.work[blockIdx.x];
  const int b = w.x, kvh = w.y, rb = w.z;
  const int seq0 = a.cu[b];
  const int n = a.cu[b + 1] - seq0;
  const int g = a.g;
  const int nrows = n * g;
  const int row = rb * F_ROWS + threadIdx.x;
  const bool valid = row < nrows;
  const int pos = valid ? row / g : n;
  const int hq = kvh * g + (valid ? row % g : 0);

  float q[D], o[D];
  const float* qp = a.q + (int64_t(seq0 + (valid ? pos : 0)) * a.hq + hq) * D;
#pragma unroll
  for (int e = 0; e < D; ++e) {
    q[e] = valid ? qp[e] : 0.f;
    o[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int pos_lo = (rb * F_ROWS) / g;
  const int first = pos_lo + (a.inclusive ? 0 : 1);
  const int t_begin = first / F_BN;
  const int t_end = (n + F_BN - 1) / F_BN;
  const float* kb = reinterpret_cast<const float*>(a.k.base);
  const float* vb = reinterpret_cast<const float*>(a.v.base);

  for (int t = t_begin; t < t_end; ++t) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < F_BN * D; idx += F_ROWS) {
      const int r = idx / D, e = idx % D;
      const int key = t * F_BN + r;
      float kv = 0.f, vv = 0.f;
      if (key < n) {
        kv = kb[kv_off<PAGED>(a.k, b, a.layer, kvh, key) + e];
        vv = vb[kv_off<PAGED>(a.v, b, a.layer, kvh, key) + e];
      }
      Ks[r][e] = kv;
      Vs[r][e] = vv;
    }
    __syncthreads();
    for (int r = 0; r < F_BN; ++r) {
      const int key = t * F_BN + r;
      const bool ok = key < n && (a.inclusive ? key >= pos : key > pos);
      if (!ok) continue;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) dot = fmaf(q[e], Ks[r][e], dot);
      const float sc = dot * a.scale;
      const float m_new = fmaxf(m, sc);
      const float corr = expf(m - m_new);
      const float p = expf(sc - m_new);
      l = l * corr + p;
#pragma unroll
      for (int e = 0; e < D; ++e) o[e] = fmaf(p, Vs[r][e], o[e] * corr);
      m = m_new;
    }
  }
  if (valid) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
    float* op = a.o + (int64_t(seq0 + pos) * a.hq + hq) * D;
#pragma unroll
    for (int e = 0; e < D; ++e) op[e] = o[e] * inv;
  }
}

template <class Args>
void fill_common(Args& x, const AttnLaunch& a) {
  x.cu = a.cu_d;
  x.work = a.work_d;
  x.k = a.k;
  x.v = a.v;
  x.layer = a.layer;
  x.hq = a.n_heads_q;
  x.g = a.n_heads_q / a.n_heads_kv;
  x.inclusive = a.inclusive;
}

}  // namespace

int attention_rows_per_item(int dtype, int head_dim) {
  (void)head_dim;
  return dtype == CC_BF16 ? ROWS : F_ROWS;
}

hipError_t launch_attention(const AttnLaunch& a, hipStream_t s) {
  if (a.n_work == 0) return hipSuccess;
  if (a.dtype == CC_BF16) {
    AttnArgs x;
    fill_common(x, a);
    x.q = static_cast<const u16*>(a.q);
    x.o = static_cast<u16*>(a.o);
    x.c2 = a.scale * kLog2e;
    if (a.paged)
      hipLaunchKernelGGL(attn_cc_bf16<true>, dim3(a.n_work), dim3(256), 0, s, x);
    else
      hipLaunchKernelGGL(attn_cc_bf16<false>, dim3(a.n_work), dim3(256), 0, s, x);
    return hipGetLastError();
  }
  AttnArgsF x;
  fill_common(x, a);
  x.q = static_cast<const float*>(a.q);
  x.o = static_cast<float*>(a.o);
  x.scale = a.scale;
  if (a.head_dim == 64) {
    if (a.paged)
      hipLaunchKernelGGL((attn_cc_f32<64, true>), dim3(a.n_work), dim3(F_ROWS), 0, s, x);
    else
      hipLaunchKernelGGL((attn_cc_f32<64, false>), dim3(a.n_work), dim3(F_ROWS), 0, s, x);
  } else {
    if (a.paged)
      hipLaunchKernelGGL((attn_cc_f32<128, true>), dim3(a.n_work), dim3(F_ROWS), 0, s, x);
    else
      hipLaunchKernelGGL((attn_cc_f32<128, false>), dim3(a.n_work), dim3(F_ROWS), 0, s, x);
  }
  return hipGetLastError();
}

}  // namespace cc
