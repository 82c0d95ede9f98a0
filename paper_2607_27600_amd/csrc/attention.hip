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
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int BN = 64;            // keys per tile
constexpr int HD = 128;           // head dim of the MFMA path
constexpr int ROWS_W = 32;        // rows per wave
constexpr int NWAVES = 4;
constexpr int ROWS = ROWS_W * NWAVES;
constexpr int KS = HD + 8;        // LDS row stride of K (elements): 272 B
constexpr int VS = BN + 8;        // LDS row stride of V^T (elements): 144 B
constexpr int K_TILE = BN * KS;
constexpr int V_TILE = HD * VS;

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
  __shared__ __attribute__((aligned(16))) u16 lds[2 * (K_TILE + V_TILE)];

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
  const int wlast = row0 + wave * ROWS_W + ROWS_W - 1;
  const int pos_hi_w = wlast < nrows ? wlast / g : n;   // invalid rows need masking always
  const int first_key = pos_lo + (a.inclusive ? 0 : 1);
  const int t_begin = first_key / BN;
  const int t_end = (n + BN - 1) / BN;

  const u16* kbase = reinterpret_cast<const u16*>(a.k.base);
  const u16* vbase = reinterpret_cast<const u16*>(a.v.base);

  // global -> register staging of one K/V tile
  // K: thread owns 16-byte column chunk kc of rows kr0 + 16*i.
  const int kc = tid & 15, kr0 = tid >> 4;
  // V: thread owns keys 4*vg .. 4*vg+3, dims 8*vd .. 8*vd+7.
  const int vg = tid & 15, vd = tid >> 4;
  uint4 kreg[4], vreg[4];

  auto load_tile = [&](int t) {
    const int key0 = t * BN;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = key0 + kr0 + 16 * i;
      if (key < n) {
        kreg[i] = ld16(kbase + kv_off<PAGED>(a.k, b, a.layer, kvh, key) + kc * 8);
      } else {
        kreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = key0 + 4 * vg + i;
      if (key < n) {
        vreg[i] = ld16(vbase + kv_off<PAGED>(a.v, b, a.layer, kvh, key) + vd * 8);
      } else {
        vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };

  // position of key 4*vg within the permuted V^T row (see the PV operand layout below)
  const int vpos = (vg >> 2) * 16 + (vg & 1) * 8 + ((vg >> 1) & 1) * 4;

  auto store_tile = [&](int buf) {
    u16* Kl = lds + buf * (K_TILE + V_TILE);
    u16* Vl = Kl + K_TILE;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<uint4*>(Kl + (kr0 + 16 * i) * KS + kc * 8) = kreg[i];
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

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 acc[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) acc[db] = f32x16{};

  if (t_begin < t_end) {
    load_tile(t_begin);
    store_tile(0);
  }
  __syncthreads();

  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    const bool more = t + 1 < t_end;
    if (more) load_tile(t + 1);

    const u16* Kl = lds + buf * (K_TILE + V_TILE);
    const u16* Vl = Kl + K_TILE;

    // S^T[key][row] for the 64 keys of the tile: two 32-key blocks.
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const bf16x8 kf = as_bf16x8(ld16(Kl + (mb * 32 + col) * KS + ks * 16 + hi * 8));
        s[mb] = mfma32(kf, qf[ks], s[mb]);
      }
    }

    const int key0 = t * BN;
    if (key0 <= pos_hi_w || key0 + BN > n) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          const bool ok = key < n && (a.inclusive ? key >= pos : key > pos);
          if (!ok) s[mb][e] = -INFINITY;
        }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[mb][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float mc = m_use * a.c2;
    const float corr = exp2f(m_run * a.c2 - mc);
    float lsum = 0.f;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(fmaf(s[mb][e], a.c2, -mc));
        s[mb][e] = p;
        lsum += p;
      }
    l_run = l_run * corr + lsum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < 4; ++db) acc[db] *= corr;

    // P^T operand: k-step kk covers keys 16*kk .. 16*kk+15; lane half hi holds keys
    // {4hi..4hi+3, 8+4hi..8+4hi+3} of that step, i.e. S^T entries 8*(kk%2) .. +7 of block kk/2.
    bf16x8 pf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 pk;
      const int mb = kk >> 1, e0 = (kk & 1) * 8;
      pk.x = pack_bf2(s[mb][e0 + 0], s[mb][e0 + 1]);
      pk.y = pack_bf2(s[mb][e0 + 2], s[mb][e0 + 3]);
      pk.z = pack_bf2(s[mb][e0 + 4], s[mb][e0 + 5]);
      pk.w = pack_bf2(s[mb][e0 + 6], s[mb][e0 + 7]);
      pf[kk] = as_bf16x8(pk);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8 vf = as_bf16x8(ld16(Vl + (db * 32 + col) * VS + kk * 16 + hi * 8));
        acc[db] = mfma32(vf, pf[kk], acc[db]);
      }

    if (more) store_tile(buf ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (valid) {
    u16* op = a.o + (int64_t(seq0 + pos) * a.hq + hq) * HD + hi * 4;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        uint2 o;
        o.x = pack_bf2(acc[db][jj * 4 + 0] * inv, acc[db][jj * 4 + 1] * inv);
        o.y = pack_bf2(acc[db][jj * 4 + 2] * inv, acc[db][jj * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + db * 32 + jj * 8) = o;
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
