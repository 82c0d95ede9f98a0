// Dense contractions of the scoring pass on CDNA4 MFMA.
//
//   y = x W^T          the layer's output projection of the fast variant (Sec. 3.1)
//   LM head + LSE      z = W_lm u for every cached entry, reduced on the fly to a
//                      per-(entry, vocabulary tile) pair (max z, sum exp(z - max)) and
//                      the target logit z[x_i]; a combine kernel turns these into
//                      logsumexp(z) - z[x_i] (Eq. (5) read as -log P).  The [N][V] logits
//                      never leave registers.
//
// bf16 kernel: C[m][n] = sum_k A[m][k] B[n][k] with both operands K-contiguous, a 256x256
// workgroup tile, 4 waves each owning a 128x128 sub-tile as 4x4 blocks of the 32x32x16
// bf16 MFMA (fp32 accumulate), K staged 64 at a time through double-buffered LDS with a
// padded row stride (144 B) so the 16-byte fragment reads of 8 consecutive rows hit
// distinct banks.  For the LM head the vocabulary is the MFMA row (M) dimension, so each
// lane holds 64 logits of one entry and the reduction over the vocabulary is mostly
// in-lane.  Tiles are rasterised entry-tile-fastest so consecutive workgroups share one
// LM-head tile.
// fp32 kernel: a plain LDS-tiled FMA GEMM with the same two epilogues.
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int GBM = 256, GBN = 256, GBK = 64;
constexpr int WGM = 2, WGN = 2, GNT = WGM * WGN * 64;
constexpr int GTM = GBM / WGM, GTN = GBN / WGN;      // 128 x 128 per wave
constexpr int GMB = GTM / 32, GNB = GTN / 32;        // 4 x 4 MFMA blocks
constexpr int GLS = GBK + 8;                         // LDS row stride (elements)

struct GemmArgs {
  const u16* A;
  const u16* B;
  int M, N, K;
  int64_t lda, ldb;
  int tiles_m, tiles_n;
  const u16* A2;   // gated loader: logical A rows alternate in blocks of 32 between A and A2
};

__device__ __forceinline__ uint4 ld16(const u16* p) { return *reinterpret_cast<const uint4*>(p); }

struct EpiStore {
  u16* out;
  int64_t ldo;
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    (void)tm;
    (void)lds;
    const int hi = lane >> 5, col = lane & 31;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int n = n0w + nb * 32 + col;
        if (n >= g.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          if (m < g.M) out[int64_t(m) * ldo + n] = f2bf(acc[mb][nb][e]);
        }
      }
  }
};

// M = vocabulary, N = cached entries.  Writes partial[tm * N + n] = (max, sumexp) over
// the workgroup's 256 vocabulary rows, and target[n] when ids[n] falls in them.
struct EpiLse {
  float2* partial;
  float* target;
  const int32_t* ids;
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    const int hi = lane >> 5, col = lane & 31;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    float2* red = reinterpret_cast<float2*>(lds);   // [WGM][GBN] pairs
    __syncthreads();   // LDS tiles are no longer read
    int id[GNB];
    float mx[GNB], sm[GNB];
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      const int n = n0w + nb * 32 + col;
      id[nb] = n < g.N ? ids[n] : -1;
      mx[nb] = -INFINITY;
      sm[nb] = 0.f;
    }
    // pass 1: per-entry max over this lane's vocabulary rows, and the target logit
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
        const bool mv = m < g.M;
#pragma unroll
        for (int nb = 0; nb < GNB; ++nb) {
          const float z = acc[mb][nb][e];
          mx[nb] = mv ? fmaxf(mx[nb], z) : mx[nb];
          if (m == id[nb]) target[n0w + nb * 32 + col] = z;
        }
      }
    // pass 2: sum of exp(z - max)
    float mc[GNB];
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) mc[nb] = mx[nb] * kLog2e;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
        const bool mv = m < g.M;
#pragma unroll
        for (int nb = 0; nb < GNB; ++nb) {
          const float t = exp2f(fmaf(acc[mb][nb][e], kLog2e, -mc[nb]));
          sm[nb] += mv ? t : 0.f;
        }
      }
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      // combine the two lane halves (rows 4*hi..)
      const float mx2 = __shfl_xor(mx[nb], 32);
      const float sm2 = __shfl_xor(sm[nb], 32);
      const float M = fmaxf(mx[nb], mx2);
      float S = 0.f;
      if (M != -INFINITY)
        S = sm[nb] * exp2f((mx[nb] - M) * kLog2e) + sm2 * exp2f((mx2 - M) * kLog2e);
      if (hi == 0) red[wm * GBN + wn * GTN + nb * 32 + col] = make_float2(M, S);
    }
    __syncthreads();
    // waves of row wm == 0 combine across the WGM row groups and write out
    if (wm == 0 && hi == 0) {
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int c = wn * GTN + nb * 32 + col;
        const int n = n0w + nb * 32 + col;
        float M = -INFINITY;
#pragma unroll
        for (int r = 0; r < WGM; ++r) M = fmaxf(M, red[r * GBN + c].x);
        float S = 0.f;
        if (M != -INFINITY) {
#pragma unroll
          for (int r = 0; r < WGM; ++r) {
            const float2 p = red[r * GBN + c];
            S += p.y * exp2f((p.x - M) * kLog2e);
          }
        }
        if (n < g.N) partial[int64_t(tm) * g.N + n] = make_float2(M, S);
      }
    }
  }
};

// M = query-projection rows (head-major, head_dim 128), N = entries.  Applies the
// rotate-half rotary embedding at each entry's position (pairs (e, e+64) of a head are
// blocks mb and mb+2 of the same lane: a wave's 128 rows are exactly one head) and
// stores q[n][m] as bf16, token-major.
struct EpiRope {
  u16* out;            // [N][M]
  const float2* rot;   // [N][64] (cos, sin) of position * theta^(-2e/128)
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    (void)tm;
    (void)lds;
    const int hi = lane >> 5, col = lane & 31;
    if (m0w >= g.M) return;
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      const int n = n0w + nb * 32 + col;
      if (n >= g.N) continue;
      u16* orow = out + int64_t(n) * g.M + m0w;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          float lo[4], up[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int e = mb * 32 + jj * 8 + hi * 4 + i;   // 0..63
            const float2 cs = rot[int64_t(n) * 64 + e];
            const float a = acc[mb][nb][jj * 4 + i], b = acc[mb + 2][nb][jj * 4 + i];
            lo[i] = a * cs.x - b * cs.y;
            up[i] = b * cs.x + a * cs.y;
          }
          const int e0 = mb * 32 + jj * 8 + hi * 4;
          uint2 v;
          v.x = pack_bf2(lo[0], lo[1]);
          v.y = pack_bf2(lo[2], lo[3]);
          *reinterpret_cast<uint2*>(orow + e0) = v;
          v.x = pack_bf2(up[0], up[1]);
          v.y = pack_bf2(up[2], up[3]);
          *reinterpret_cast<uint2*>(orow + e0 + 64) = v;
        }
    }
  }
};

// M = entries, N = model width: the fp32 residual stream takes h[m][n] += acc.
struct EpiResidual {
  float* h;   // [M][N]
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    (void)tm;
    (void)lds;
    const int hi = lane >> 5, col = lane & 31;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int n = n0w + nb * 32 + col;
        if (n >= g.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          if (m < g.M) h[int64_t(m) * g.N + n] += acc[mb][nb][e];
        }
      }
  }
};

// M = interleaved gate/up rows (see the gated loader), N = entries:
// act[n][f] = silu(gate) * up, bf16, token-major [N][F].
struct EpiSwiglu {
  u16* act;
  int F;
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    (void)tm;
    (void)lds;
    const int hi = lane >> 5, col = lane & 31;
#pragma unroll
    for (int pr = 0; pr < GMB / 2; ++pr) {
      const int r0 = m0w + pr * 64;            // logical row of this gate block
      if (r0 >= g.M) continue;
      const int f0 = (r0 >> 6) * 32;
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int n = n0w + nb * 32 + col;
        if (n >= g.N) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float gt = acc[2 * pr][nb][jj * 4 + i];
            const float up = acc[2 * pr + 1][nb][jj * 4 + i];
            o[i] = gt / (1.f + expf(-gt)) * up;
          }
          uint2 v;
          v.x = pack_bf2(o[0], o[1]);
          v.y = pack_bf2(o[2], o[3]);
          *reinterpret_cast<uint2*>(act + int64_t(n) * F + f0 + jj * 8 + hi * 4) = v;
        }
      }
    }
  }
};

// Workgroup -> output tile.  Workgroups are dispatched round-robin over the 8 XCDs (each
// with its own L2), so consecutive logical tiles are first given to one XCD, then the
// logical order walks groups of GROUP_M tile rows with the row index fastest: the ~32
// workgroups an XCD runs at once cover a 4 x 8 block of tiles and share their A and B
// k-slices in that XCD's L2.
constexpr int GROUP_M = 4;

__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int T = tiles_m * tiles_n;
  const int per = T / 8, rem = T % 8;
  const int x = bid % 8, j = bid / 8;
  const int L = x * per + min(x, rem) + j;
  const int group = L / (GROUP_M * tiles_n);
  const int first = group * GROUP_M;
  const int gsize = min(GROUP_M, tiles_m - first);
  const int within = L - group * GROUP_M * tiles_n;
  tm = first + within % gsize;
  tn = within / gsize;
}

// Scheduling hints: interleave MFMAs with LDS reads / writes / global loads so the matrix
// pipe stays busy while the wave issues its memory traffic.
#define SCHED_MFMA 0x008
#define SCHED_VMEM_READ 0x020
#define SCHED_DS_READ 0x100
#define SCHED_DS_WRITE 0x200

template <class Epi, bool GATED = false>
__global__ __launch_bounds__(GNT, 1) void gemm_tn_bf16(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(16))) u16 lds[2 * (GBM + GBN) * GLS];
  int tm, tn;
  tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn);
  const int m0 = tm * GBM, n0 = tn * GBN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hi = lane >> 5, col = lane & 31;
  const int wm = wave / WGN, wn = wave % WGN;

  constexpr int RA = GBM * 8 / GNT, RB = GBN * 8 / GNT, RSTEP = GNT / 8;
  const int lc = tid & 7, lr = tid >> 3;
  // Rows past the matrix edge are clamped to the last row: their products land in output
  // rows/columns the epilogues discard, so no zero fill (and no branch) is needed.
  const u16* pa[RA];
  const u16* pb[RB];
#pragma unroll
  for (int i = 0; i < RA; ++i) {
    const int r = min(m0 + lr + RSTEP * i, g.M - 1);
    if constexpr (GATED) {
      // rows [64j, 64j+32) are W_gate rows [32j, 32j+32), rows [64j+32, 64j+64) the same
      // W_up rows, so each wave's 32-row MFMA blocks pair gate and up for one column range
      const u16* base = ((r >> 5) & 1) ? g.A2 : g.A;
      pa[i] = base + int64_t((r >> 6) * 32 + (r & 31)) * g.lda + lc * 8;
    } else {
      pa[i] = g.A + int64_t(r) * g.lda + lc * 8;
    }
  }
#pragma unroll
  for (int i = 0; i < RB; ++i)
    pb[i] = g.B + int64_t(min(n0 + lr + RSTEP * i, g.N - 1)) * g.ldb + lc * 8;
  uint4 ra[RA], rbv[RB];

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < RA; ++i) ra[i] = ld16(pa[i] + k0);
#pragma unroll
    for (int i = 0; i < RB; ++i) rbv[i] = ld16(pb[i] + k0);
  };
  auto lstore = [&](int buf) {
    u16* As = lds + buf * (GBM + GBN) * GLS;
    u16* Bs = As + GBM * GLS;
#pragma unroll
    for (int i = 0; i < RA; ++i)
      *reinterpret_cast<uint4*>(As + (lr + RSTEP * i) * GLS + lc * 8) = ra[i];
#pragma unroll
    for (int i = 0; i < RB; ++i)
      *reinterpret_cast<uint4*>(Bs + (lr + RSTEP * i) * GLS + lc * 8) = rbv[i];
  };
  auto fread = [&](int buf, int ks, bf16x8 (&fa)[GMB], bf16x8 (&fb)[GNB]) {
    const u16* As = lds + buf * (GBM + GBN) * GLS;
    const u16* Bs = As + GBM * GLS;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
      fa[mb] = as_bf16x8(ld16(As + (wm * GTM + mb * 32 + col) * GLS + ks * 16 + hi * 8));
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb)
      fb[nb] = as_bf16x8(ld16(Bs + (wn * GTN + nb * 32 + col) * GLS + ks * 16 + hi * 8));
  };

  f32x16 acc[GMB][GNB];
#pragma unroll
  for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) acc[mb][nb] = f32x16{};
  auto mfmas = [&](const bf16x8 (&fa)[GMB], const bf16x8 (&fb)[GNB]) {
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) acc[mb][nb] = mfma32(fa[mb], fb[nb], acc[mb][nb]);
  };

  const int nk = g.K / GBK;
  bf16x8 fa0[GMB], fb0[GNB], fa1[GMB], fb1[GNB];
  gload(0);
  lstore(0);
  __syncthreads();
  fread(0, 0, fa0, fb0);
  if (nk > 1) gload(GBK);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    // k-step 0: read step-1 fragments while the step-0 MFMAs run
    __builtin_amdgcn_sched_barrier(0);
    fread(buf, 1, fa1, fb1);
    mfmas(fa0, fb0);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
    // k-step 1
    fread(buf, 2, fa0, fb0);
    mfmas(fa1, fb1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 8, 0);
    __builtin_amdgcn_sched_barrier(0);
    // k-step 2, then the next tile goes from registers to the other LDS buffer
    fread(buf, 3, fa1, fb1);
    mfmas(fa0, fb0);
    lstore(buf ^ 1);   // on the last tile this fills a buffer nobody reads
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_WRITE, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // k-step 3: fragments of the next tile's step 0 and the global loads two tiles ahead
    // are issued between the MFMAs
    fread(buf ^ 1, 0, fa0, fb0);
    gload(min(kt + 2, nk - 1) * GBK);   // past the end: a harmless reload of the last tile
    mfmas(fa1, fb1);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_VMEM_READ, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  __syncthreads();
  epi(acc, g, tm, m0 + wm * GTM, n0 + wn * GTN, lane, lds);
}

// ------------------------------------------------------------------ fp32 path

constexpr int FT = 64, FK = 16;

struct GemmArgsF {
  const float* A;
  const float* B;
  int M, N, K;
  int64_t lda, ldb;
  int tiles_n;
};

struct EpiStoreF {
  float* out;
  int64_t ldo;
  __device__ void operator()(const float (&c)[4][4], const GemmArgsF& g, int tm, int m0, int n0,
                             float* lds) const {
    (void)tm;
    (void)lds;
    const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
        if (m < g.M && n < g.N) out[int64_t(m) * ldo + n] = c[i][j];
      }
  }
};

struct EpiLseF {
  float2* partial;
  float* target;
  const int32_t* ids;
  __device__ void operator()(const float (&c)[4][4], const GemmArgsF& g, int tm, int m0, int n0,
                             float* lds) const {
    const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
    float* T = lds;   // [FT][FT + 1], T[m][n]
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) T[(ty * 4 + i) * (FT + 1) + tx * 4 + j] = c[i][j];
    __syncthreads();
    if (threadIdx.x < FT) {
      const int nl = threadIdx.x, n = n0 + nl;
      if (n < g.N) {
        const int id = ids[n];
        float mx = -INFINITY;
        for (int ml = 0; ml < FT && m0 + ml < g.M; ++ml) {
          const float z = T[ml * (FT + 1) + nl];
          mx = fmaxf(mx, z);
          if (m0 + ml == id) target[n] = z;
        }
        float s = 0.f;
        for (int ml = 0; ml < FT && m0 + ml < g.M; ++ml) s += expf(T[ml * (FT + 1) + nl] - mx);
        partial[int64_t(tm) * g.N + n] = make_float2(mx, s);
      }
    }
  }
};

template <class Epi>
__global__ __launch_bounds__(256) void gemm_tn_f32(GemmArgsF g, Epi epi) {
  __shared__ float lds[FT * (FT + 1)];
  float* As = lds;                 // [FK][FT + 4]
  float* Bs = lds + FK * (FT + 4); // [FK][FT + 4]
  const int tm = blockIdx.x / g.tiles_n, tn = blockIdx.x % g.tiles_n;
  const int m0 = tm * FT, n0 = tn * FT;
  const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
  float c[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += FK) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < FT * FK; idx += 256) {
      const int r = idx / FK, kk = idx % FK;
      const int m = m0 + r, n = n0 + r, k = k0 + kk;
      As[kk * (FT + 4) + r] = (m < g.M && k < g.K) ? g.A[int64_t(m) * g.lda + k] : 0.f;
      Bs[kk * (FT + 4) + r] = (n < g.N && k < g.K) ? g.B[int64_t(n) * g.ldb + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk * (FT + 4) + ty * 4 + i];
        b[i] = Bs[kk * (FT + 4) + tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) c[i][j] = fmaf(a[i], b[j], c[i][j]);
    }
  }
  epi(c, g, tm, m0, n0, lds);
}

// ------------------------------------------------------------------ LSE combine

// One workgroup per 16 entries: thread (group gi, entry e) folds the vocabulary tiles
// gi, gi+16, ... of entry e (16 consecutive entries read 128 contiguous bytes of a tile's
// row of partials), then the 16 groups are folded in LDS.
constexpr int CMB_E = 16, CMB_G = 16;

__device__ __forceinline__ void lse_fold(float& M, float& S, float m, float s) {
  if (m == -INFINITY) return;
  if (m > M) {
    S = S * expf(M - m) + s;
    M = m;
  } else {
    S += s * expf(m - M);
  }
}

__global__ __launch_bounds__(CMB_E * CMB_G) void lse_combine(const float2* partial, int n_tiles,
                                                            const float* target, const int32_t* cu,
                                                            int n_seqs, int n_frozen, int N,
                                                            float* scores, float* lse_out) {
  __shared__ float2 red[CMB_G][CMB_E];
  const int e = threadIdx.x % CMB_E, gi = threadIdx.x / CMB_E;
  const int n = blockIdx.x * CMB_E + e;
  float M = -INFINITY, S = 0.f;
  if (n < N) {
    for (int t = gi; t < n_tiles; t += CMB_G) {
      const float2 p = partial[int64_t(t) * N + n];
      lse_fold(M, S, p.x, p.y);
    }
  }
  red[gi][e] = make_float2(M, S);
  __syncthreads();
  if (gi == 0 && n < N) {
    float Mt = -INFINITY, St = 0.f;
#pragma unroll
    for (int r = 0; r < CMB_G; ++r) lse_fold(Mt, St, red[r][e].x, red[r][e].y);
    const float lse = Mt + logf(St);
    // sequence of entry n: the last b with cu[b] <= n
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= n) lo = mid; else hi = mid - 1;
    }
    const bool last = n == cu[lo + 1] - 1;
    const bool frozen = n - cu[lo] < n_frozen;
    scores[n] = (last || frozen) ? INFINITY : lse - target[n];
    if (lse_out) lse_out[n] = lse;
  }
}

}  // namespace

int lmhead_vocab_tile(int dtype) { return dtype == CC_BF16 ? GBM : FT; }

hipError_t launch_linear(int dtype, const void* x, const void* w, void* y, int M, int N, int K,
                         hipStream_t s) {
  if (M == 0 || N == 0) return hipSuccess;
  if (dtype == CC_BF16) {
    GemmArgs g;
    g.A2 = nullptr;
    g.A = static_cast<const u16*>(x);
    g.B = static_cast<const u16*>(w);
    g.M = M;
    g.N = N;
    g.K = K;
    g.lda = K;
    g.ldb = K;
    g.tiles_n = (N + GBN - 1) / GBN;
    g.tiles_m = (M + GBM - 1) / GBM;
    const int tiles = g.tiles_m * g.tiles_n;
    EpiStore e{static_cast<u16*>(y), N};
    hipLaunchKernelGGL(gemm_tn_bf16<EpiStore>, dim3(tiles), dim3(GNT), 0, s, g, e);
    return hipGetLastError();
  }
  GemmArgsF g;
  g.A = static_cast<const float*>(x);
  g.B = static_cast<const float*>(w);
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = K;
  g.ldb = K;
  g.tiles_n = (N + FT - 1) / FT;
  const int tiles = ((M + FT - 1) / FT) * g.tiles_n;
  EpiStoreF e{static_cast<float*>(y), N};
  hipLaunchKernelGGL(gemm_tn_f32<EpiStoreF>, dim3(tiles), dim3(256), 0, s, g, e);
  return hipGetLastError();
}

hipError_t launch_lmhead(const LmHeadLaunch& a, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  int n_vt;
  if (a.dtype == CC_BF16) {
    GemmArgs g;
    g.A2 = nullptr;
    g.A = static_cast<const u16*>(a.w_lm);
    g.B = static_cast<const u16*>(a.u);
    g.M = a.V;
    g.N = a.N;
    g.K = a.D;
    g.lda = a.D;
    g.ldb = a.D;
    g.tiles_n = (a.N + GBN - 1) / GBN;
    n_vt = (a.V + GBM - 1) / GBM;
    g.tiles_m = n_vt;
    EpiLse e{a.partial, a.target, a.ids};
    hipLaunchKernelGGL(gemm_tn_bf16<EpiLse>, dim3(n_vt * g.tiles_n), dim3(GNT), 0, s, g, e);
  } else {
    GemmArgsF g;
    g.A = static_cast<const float*>(a.w_lm);
    g.B = static_cast<const float*>(a.u);
    g.M = a.V;
    g.N = a.N;
    g.K = a.D;
    g.lda = a.D;
    g.ldb = a.D;
    g.tiles_n = (a.N + FT - 1) / FT;
    n_vt = (a.V + FT - 1) / FT;
    EpiLseF e{a.partial, a.target, a.ids};
    hipLaunchKernelGGL(gemm_tn_f32<EpiLseF>, dim3(n_vt * g.tiles_n), dim3(256), 0, s, g, e);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(lse_combine, dim3((a.N + CMB_E - 1) / CMB_E), dim3(CMB_E * CMB_G), 0, s,
                     a.partial, n_vt,
                     a.target, a.cu_d, a.n_seqs, a.n_frozen, a.N, a.scores, a.lse);
  return hipGetLastError();
}

namespace {
GemmArgs make_args(const void* a, const void* b, int M, int N, int K, int64_t lda, int64_t ldb) {
  GemmArgs g;
  g.A = static_cast<const u16*>(a);
  g.B = static_cast<const u16*>(b);
  g.A2 = nullptr;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.tiles_m = (M + GBM - 1) / GBM;
  g.tiles_n = (N + GBN - 1) / GBN;
  return g;
}
}  // namespace

hipError_t launch_qproj_rope(const void* wq, const void* a, void* q, const float2* rot, int N,
                             int D, int HD, hipStream_t s) {
  if (N == 0) return hipSuccess;
  GemmArgs g = make_args(wq, a, HD, N, D, D, D);
  EpiRope e{static_cast<u16*>(q), rot};
  hipLaunchKernelGGL(gemm_tn_bf16<EpiRope>, dim3(g.tiles_m * g.tiles_n), dim3(GNT), 0, s, g, e);
  return hipGetLastError();
}

hipError_t launch_linear_residual(const void* x, const void* w, float* h, int M, int N, int K,
                                  hipStream_t s) {
  if (M == 0) return hipSuccess;
  GemmArgs g = make_args(x, w, M, N, K, K, K);
  EpiResidual e{h};
  hipLaunchKernelGGL(gemm_tn_bf16<EpiResidual>, dim3(g.tiles_m * g.tiles_n), dim3(GNT), 0, s, g,
                     e);
  return hipGetLastError();
}

hipError_t launch_gate_up_swiglu(const void* w_gate, const void* w_up, const void* b, void* act,
                                 int N, int D, int F, hipStream_t s) {
  if (N == 0) return hipSuccess;
  GemmArgs g = make_args(w_gate, b, 2 * F, N, D, D, D);
  g.A2 = static_cast<const u16*>(w_up);
  EpiSwiglu e{static_cast<u16*>(act), F};
  hipLaunchKernelGGL((gemm_tn_bf16<EpiSwiglu, true>), dim3(g.tiles_m * g.tiles_n), dim3(GNT), 0,
                     s, g, e);
  return hipGetLastError();
}

}  // namespace cc
