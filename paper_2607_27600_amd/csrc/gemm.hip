// Dense contractions of the scoring pass on CDNA4 MFMA.
//
//   y = x W^T          the layer's output projection of the fast variant (Sec. 3.1)
//   LM head + LSE      z = W_lm u for every cached entry, reduced on the fly to a
//                      per-(entry, vocabulary tile) pair (max z, sum exp(z - max)); the
//                      lane that holds z[x_i] in its accumulators writes the target logit
//                      from them; a combine kernel turns these into logsumexp(z) - z[x_i]
//                      (Eq. (5) read as -log P).  The [N][V] logits never leave registers.
//
// bf16 kernel: C[m][n] = sum_k A[m][k] B[n][k] with both operands K-contiguous, a 256x256
// workgroup tile, 8 waves (two per SIMD, so one wave's barrier and load waits hide behind
// the other's MFMAs) each owning a 128x64 sub-tile as 4x2 blocks of the 32x32x16 bf16 MFMA
// (fp32 accumulate), K staged 64 at a time through two LDS stages.  For the LM head the vocabulary is the MFMA row (M) dimension, so each
// lane holds 64 logits of one entry and the reduction over the vocabulary is mostly
// in-lane.  Tiles are rasterised entry-tile-fastest so consecutive workgroups share one
// LM-head tile.
// fp32 kernel: a plain LDS-tiled FMA GEMM with the same two epilogues.
#include <algorithm>
#include <type_traits>

#include "cc_internal.h"

namespace cc {
namespace {

constexpr int GBM = 256, GBN = 256, GBK = 64;
constexpr int WGM = 2, WGN = 4, GNT = WGM * WGN * 64;   // 8 waves: two per SIMD
constexpr int NWAVE = WGM * WGN;
constexpr int LPW = 32 / NWAVE;   // 1 KB direct-load instructions per wave per operand tile
constexpr int GTM = GBM / WGM, GTN = GBN / WGN;      // 128 x 64 per wave
constexpr int GMB = GTM / 32, GNB = GTN / 32;        // 4 x 2 MFMA blocks

struct GemmArgs {
  const u16* A;
  const u16* B;
  int M, N, K;
  int64_t lda, ldb;
  int tiles_m, tiles_n;
  const u16* A2;   // gated loader: logical A rows alternate in blocks of 32 between A and A2
  int kt_split = 0;   // split-K: k-tiles per slice, slice = blockIdx.y (0: one pass over K)
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
// the workgroup's 256 vocabulary rows.  The whole epilogue runs while the matrix cores
// idle, so it is kept to one max and one exp-accumulate per logit; only workgroups on the
// vocabulary edge take the masked variant.
// Target gather: the cached token x_n of entry n lies in exactly one vocabulary tile, one
// wave row of it and one lane half; that lane writes target[n] = its accumulator for row
// x_n (times the scales below), so the target logit and the log-sum-exp come from the
// same accumulators.  The ids are loaded first and the selection runs only in waves where
// some lane owns a target (about 3% of them at a vocabulary of 128k).
// An FP8 LM head passes the dequantization scales: the logit is acc * sw * su[n]
// (su per entry, sw for the whole matrix); without them the factor is 1 and the
// arithmetic is unchanged.
struct EpiLse {
  float2* partial;
  float* target;               // [N] target logits z[x_n]
  const int32_t* ids;          // [N] cached token ids
  const float* su = nullptr;   // [N] per-entry scale, or null
  const float* sw = nullptr;   // [1] matrix scale (device), with su
  template <bool EDGE>
  __device__ __forceinline__ void reduce(const f32x16 (&acc)[GMB][GNB], int M, int m0w, int hi,
                                         const float (&f)[GNB], float (&mx)[GNB],
                                         float (&sm)[GNB]) const {
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) mx[nb] = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const bool ok = !EDGE || (m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3) < M);
#pragma unroll
        for (int nb = 0; nb < GNB; ++nb)
          if (ok) mx[nb] = fmaxf(mx[nb], acc[mb][nb][e]);
      }
    float mc[GNB], c[GNB];
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      // logits are acc * f (f >= 0), so their max is mx * f; a lane whose rows are all
      // past the edge keeps max = -inf and sum = 0
      if (mx[nb] != -INFINITY) mx[nb] *= f[nb];
      mc[nb] = mx[nb] == -INFINITY ? 0.f : mx[nb] * kLog2e;
      c[nb] = kLog2e * f[nb];
      sm[nb] = 0.f;
    }
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const bool ok = !EDGE || (m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3) < M);
#pragma unroll
        for (int nb = 0; nb < GNB; ++nb)
          if (ok) sm[nb] += fast_exp2(fmaf(acc[mb][nb][e], c[nb], -mc[nb]));
      }
  }

  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    const int hi = lane >> 5, col = lane & 31;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    float2* red = reinterpret_cast<float2*>(lds);   // [WGM][GBN] pairs
    // target rows relative to this wave's first vocabulary row (loaded before the
    // reduction so their latency hides behind it)
    int rt[GNB];
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) rt[nb] = ids[min(n0w + nb * 32 + col, g.N - 1)] - m0w;
    float f[GNB];
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb)
      f[nb] = su ? sw[0] * su[min(n0w + nb * 32 + col, g.N - 1)] : 1.f;
    float mx[GNB], sm[GNB];
    if (tm * GBM + GBM <= g.M)
      reduce<false>(acc, g.M, m0w, hi, f, mx, sm);
    else
      reduce<true>(acc, g.M, m0w, hi, f, mx, sm);
    // row r of the wave's 128 sits in block r / 32, element 4 ((r % 32) / 8) + r % 4 of the
    // lane half (r / 4) % 2
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      const int r = rt[nb];
      const bool own = n0w + nb * 32 + col < g.N && uint32_t(r) < uint32_t(GTM) &&
                       ((r >> 2) & 1) == hi;
      if (__any(own)) {
        const int idx = (r >> 5) * 16 + ((r & 31) >> 3) * 4 + (r & 3);
        float z = 0.f;
#pragma unroll
        for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
          for (int e = 0; e < 16; ++e) z = idx == mb * 16 + e ? acc[mb][nb][e] : z;
        if (own) target[n0w + nb * 32 + col] = z * f[nb];
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
    // Per 32-row block: the 16 x GNB residual values are loaded together (rows and columns
    // clamped, so no load is conditional), then added and stored.  Element by element, each
    // add waited for its own load: 128 memory round trips per lane.
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb) {
      float r[GNB][16];
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int nc = min(n0w + nb * 32 + col, g.N - 1);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = min(m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3), g.M - 1);
          r[nb][e] = h[int64_t(m) * g.N + nc];
        }
      }
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int n = n0w + nb * 32 + col;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = m0w + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          if (n < g.N && m < g.M) h[int64_t(m) * g.N + n] = r[nb][e] + acc[mb][nb][e];
        }
      }
    }
  }
};

// Split-K: one K slice's fp32 products, part[slice][m][n] (NM = false, the layout of the
// residual stream) or part[slice][n][m] (NM = true, the token-major layout of the query
// projection).  A reduce kernel sums the slices in order and applies the real epilogue.
template <bool NM>
struct EpiPartial {
  float* part;
  __device__ void operator()(const f32x16 (&acc)[GMB][GNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    (void)tm;
    (void)lds;
    const int hi = lane >> 5, col = lane & 31;
    float* p = part + int64_t(blockIdx.y) * g.M * g.N;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < GNB; ++nb) {
        const int n = n0w + nb * 32 + col;
        if (n >= g.N) continue;
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
          const int m = m0w + mb * 32 + e4 * 8 + hi * 4;   // rows m .. m+3 of this lane
          if constexpr (NM) {
            // M is a multiple of 4 here (whole heads), so the four rows go out as one float4
            if (m < g.M)
              *reinterpret_cast<float4*>(p + int64_t(n) * g.M + m) =
                  make_float4(acc[mb][nb][4 * e4], acc[mb][nb][4 * e4 + 1],
                              acc[mb][nb][4 * e4 + 2], acc[mb][nb][4 * e4 + 3]);
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (m + i < g.M) p[int64_t(m + i) * g.N + n] = acc[mb][nb][4 * e4 + i];
          }
        }
      }
  }
};

// Split-K sum into the fp32 residual stream: h[i] += part[0][i] + ... + part[S-1][i]
// (count a multiple of 4).
__global__ __launch_bounds__(256) void reduce_residual(const float* __restrict__ part, int S,
                                                       int64_t count, float* __restrict__ h) {
  const int64_t i = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i >= count) return;
  float4 t = *reinterpret_cast<const float4*>(part + i);
  for (int sl = 1; sl < S; ++sl) {
    const float4 v = *reinterpret_cast<const float4*>(part + int64_t(sl) * count + i);
    t.x += v.x;
    t.y += v.y;
    t.z += v.z;
    t.w += v.w;
  }
  float4 r = *reinterpret_cast<const float4*>(h + i);
  r.x += t.x;
  r.y += t.y;
  r.z += t.z;
  r.w += t.w;
  *reinterpret_cast<float4*>(h + i) = r;
}

// Split-K query projection: q = the sum of the slices (part [S][N][M]), then the rotate-half
// rotary embedding of EpiRope at each entry's position, stored as bf16 [N][M].  One thread
// per (entry, head, pair e of 0..63); head_dim 128.
__global__ __launch_bounds__(256) void reduce_rope(const float* __restrict__ part, int S, int N,
                                                   int M, const float2* __restrict__ rot,
                                                   u16* __restrict__ q) {
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int half = M / 2;
  if (t >= int64_t(N) * half) return;
  const int n = int(t / half), r = int(t % half);
  const int e = r & 63, m = (r >> 6) * 128 + e;
  const int64_t cnt = int64_t(N) * M, o = int64_t(n) * M + m;
  float a = part[o], b = part[o + 64];
  for (int sl = 1; sl < S; ++sl) {
    a += part[sl * cnt + o];
    b += part[sl * cnt + o + 64];
  }
  const float2 cs = rot[int64_t(n) * 64 + e];
  q[o] = f2bf(a * cs.x - b * cs.y);
  q[o + 64] = f2bf(b * cs.x + a * cs.y);
}

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

// Workgroup -> output tile.  The tile grid is cut into supertiles of ST_M x ST_N tiles (rows
// of supertiles first, each row walked left to right), and inside a supertile the workgroups
// walk groups of GROUP_M tile rows with the row index fastest.  Workgroups are dealt to the
// eight XCDs round robin, so each XCD's resident workgroups cover GROUP_M rows x 8 columns
// of tiles (few distinct k-slices per k-step in its L2), and the whole chip works inside one
// supertile at a time, whose operand rows (64 + 16 tiles of 256 rows, 147 MB at a 3584-wide
// K) stay in the Infinity Cache while the supertile row is swept: the wide operand is then
// re-read once per supertile row instead of once per GROUP_M tile rows.  A grid of at most 16
// tile columns is the plain GROUP_M walk.  (Partitioning the order by XCD explicitly measured
// no better; 64 supertile rows measured 1.4% faster than 32 on the 152064 x 75696 LM head,
// 96 and 128 no better than 64.)
constexpr int GROUP_M = 4;
constexpr int ST_M = 64, ST_N = 16;

__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int sr = bid / (ST_M * tiles_n);
  const int rem = bid - sr * (ST_M * tiles_n);
  const int m0 = sr * ST_M;
  const int sm = min(ST_M, tiles_m - m0);        // tile rows in this supertile row
  const int sc = rem / (sm * ST_N);
  const int rem2 = rem - sc * (sm * ST_N);
  const int n0 = sc * ST_N;
  const int sn = min(ST_N, tiles_n - n0);        // tile columns in this supertile
  const int group = rem2 / (GROUP_M * sn);
  const int first = group * GROUP_M;
  const int gsize = min(GROUP_M, sm - first);
  const int within = rem2 - group * (GROUP_M * sn);
  tm = m0 + first + within % gsize;
  tn = n0 + within / gsize;
}

// Scheduling hints: interleave MFMAs with LDS reads / writes / global loads so the matrix
// pipe stays busy while the wave issues its memory traffic.
#define SCHED_MFMA 0x008
#define SCHED_VMEM 0x010
#define SCHED_DS_READ 0x100
#define SCHED_DS_WRITE 0x200

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_void;
constexpr int STAGE = (GBM + GBN) * GBK;   // bf16 elements per LDS stage (64 KB)

// The main loop.  Operand tiles go from global memory straight into LDS
// (global_load_lds_dwordx4: lane i of a wave instruction fills bytes 16i..16i+15 of a 1 KB
// run), so no registers stage them and no LDS write instructions are issued.  Tiles are
// unpadded [rows][64] bf16 with the 16-byte chunk c of row r stored at chunk
// c ^ ((r >> 1) & 7).  The LDS serves a 16-byte read for 16 lanes at a time across 64
// banks (256 B); the fragment reads of 16 consecutive rows at one chunk then cover all 64
// banks exactly once (two 128-byte rows per bank cycle, the XOR spreading the 8 even and
// the 8 odd rows over the 8 chunk slots).  Two
// stages are distinct LDS objects so the compiler can tell the stage being filled from the
// stage being read (a shared object would make it wait for the loads before every read).
// One barrier per k-tile, placed after the step-3 fragments are read: past it, the next
// stage is complete and the current one is free for the loads of the tile after next.
// Each stage is loaded in two halves issued between MFMAs (see the loop below).
template <class Epi, bool GATED = false>
__global__ __launch_bounds__(GNT, 1) void gemm_tn_bf16(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) u16 lds0[STAGE];
  __shared__ __attribute__((aligned(1024))) u16 lds1[STAGE];
  int tm, tn;
  tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn);
  const int m0 = tm * GBM, n0 = tn * GBN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hi = lane >> 5, col = lane & 31;
  const int wm = wave / WGN, wn = wave % WGN;
  // split-K: this workgroup's slice covers k-tiles kt0 .. kt0 + nk - 1
  const int kt0 = g.kt_split ? int(blockIdx.y) * g.kt_split : 0;
  const int nk = g.kt_split ? min(g.kt_split, g.K / GBK - kt0) : g.K / GBK;

  // wave w, load instruction j covers tile rows (8w + j) * 8 .. +8; rows past the matrix
  // edge are clamped to the last row (their products land in outputs the epilogues
  // discard), so the loop has no branches
  const u16* ga[LPW];
  const u16* gb[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int r = (wave * LPW + j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    const int ra = min(m0 + r, g.M - 1);
    if constexpr (GATED) {
      // rows [64i, 64i+32) are W_gate rows [32i, 32i+32), rows [64i+32, 64i+64) the same
      // W_up rows, so each wave's 32-row MFMA blocks pair gate and up for one column range
      const u16* base = ((ra >> 5) & 1) ? g.A2 : g.A;
      ga[j] = base + int64_t((ra >> 6) * 32 + (ra & 31)) * g.lda + c * 8 + kt0 * GBK;
    } else {
      ga[j] = g.A + int64_t(ra) * g.lda + c * 8 + kt0 * GBK;
    }
    gb[j] = g.B + int64_t(min(n0 + r, g.N - 1)) * g.ldb + c * 8 + kt0 * GBK;
  }
  // Half h of a stage: h = 0 the A rows, h = 1 the B rows (LPW direct loads per wave).
  auto issue_half = [&](u16* stage, int k0, int h) {
    u16* base = stage + wave * LPW * 512 + h * GBM * GBK;
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      __builtin_amdgcn_global_load_lds((global_void*)((h ? gb[j] : ga[j]) + k0),
                                       (lds_void*)(base + j * 512), 16, 0, 0);
  };
  auto fread = [&](const u16* As, int ks, bf16x8 (&fa)[GMB], bf16x8 (&fb)[GNB]) {
    const u16* Bs = As + GBM * GBK;
    const int c = 2 * ks + hi;
#pragma unroll
    for (int mb = 0; mb < GMB; ++mb) {
      const int r = wm * GTM + mb * 32 + col;
      fa[mb] = as_bf16x8(ld16(As + r * GBK + ((c ^ ((r >> 1) & 7)) * 8)));
    }
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) {
      const int r = wn * GTN + nb * 32 + col;
      fb[nb] = as_bf16x8(ld16(Bs + r * GBK + ((c ^ ((r >> 1) & 7)) * 8)));
    }
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
  // scheduling hint: one fragment read between consecutive MFMAs, then the rest
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < GMB + GNB; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, GMB * GNB - (GMB + GNB), 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  // the same, with one direct load after every other MFMA
  auto interleave_loads = [&]() {
#pragma unroll
    for (int i = 0; i < GMB * GNB; ++i) {
      __builtin_amdgcn_sched_group_barrier(SCHED_MFMA, 1, 0);
      if (i < GMB + GNB) __builtin_amdgcn_sched_group_barrier(SCHED_DS_READ, 1, 0);
      if ((i & 1) == 0) __builtin_amdgcn_sched_group_barrier(SCHED_VMEM, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  bf16x8 fa0[GMB], fb0[GNB], fa1[GMB], fb1[GNB];
  // One k-tile from `cur`; fragments of each step are read during the previous step.  The
  // loads of a stage are split in two halves issued between MFMAs, never in one burst: when
  // every wave of the CU issues its loads at once they queue on the memory pipeline and the
  // waves stall behind them.  The B half of `nxt` (k-tile kt+1) goes out during the first
  // step; the A half of `cur` (k-tile kt+2, past the end: a reload) right after the barrier
  // that frees `cur`.
  auto tile = [&](const u16* cur, u16* nxt, int kt) {
    __builtin_amdgcn_sched_barrier(0);
    fread(cur, 1, fa1, fb1);
    mfmas(fa0, fb0);
    issue_half(nxt, min(kt + 1, nk - 1) * GBK, 1);
    interleave_loads();
    fread(cur, 2, fa0, fb0);
    mfmas(fa1, fb1);
    interleave();
    fread(cur, 3, fa1, fb1);
    mfmas(fa0, fb0);
    interleave();
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads into `nxt` have landed
    __syncthreads();                 // everyone's have, and everyone is done with `cur`
    issue_half(const_cast<u16*>(cur), min(kt + 2, nk - 1) * GBK, 0);
    fread(nxt, 0, fa0, fb0);
    mfmas(fa1, fb1);
    interleave_loads();
  };
  issue_half(lds0, 0, 0);
  issue_half(lds0, 0, 1);
  issue_half(lds1, min(1, nk - 1) * GBK, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  fread(lds0, 0, fa0, fb0);
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    tile(lds0, lds1, kt);
    tile(lds1, lds0, kt + 1);
  }
  if (kt < nk) tile(lds0, lds1, kt);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  epi(acc, g, tm, m0 + wm * GTM, n0 + wn * GTN, lane, lds0);
}

// ------------------------------------------------------------------ packed LM head
// The same contraction with both operands stored as the LDS images the kernel stages.  A
// [R][K] matrix is packed per 256-row tile and 32-wide k-step into one 16 KB block: row r of
// the tile at bytes 64r .. 64r+63, its 16-byte chunk c (k = 8c .. 8c+7 of the step) at
// chunk position c ^ ((r >> 1) & 3); rows past R are zero.  Staging a block is then a
// contiguous 16 KB copy (one 1 KB run per wave instruction), which the memory system
// delivers markedly faster than 256 row pieces of 64 bytes.  The XOR on row bits 1-2 keeps
// the 16-byte fragment reads free of bank conflicts: measured on gfx950, the same reads
// with the chunk swizzled by row bits 2-3 (or not at all) conflict two ways and run at half
// the LDS rate.  The vocabulary weight is packed once per model, the entry rows at every
// call.
//
// Matrix cores: 16x16x32 bf16 MFMA (lane l reads row l%16 of a 16-row block at chunk l/16;
// it holds rows 4(l/16) .. +3 of column l%16 of the result), 8 waves of 128x64 as 8x4
// blocks.  Four stages of one k-step each: the loads of k-step t+3 are issued while k-step
// t is multiplied, so a load has three k-steps to land.
constexpr int PK_ROWS = 256, PK_K = 32;
constexpr int PK_BLOCK = PK_ROWS * PK_K;          // elements per packed block (16 KB)
constexpr int PSTAGE = 2 * PK_BLOCK;              // an A block and a B block (32 KB)
constexpr int PNST = 4;                           // stages
constexpr int HMB = GTM / 16, HNB = GTN / 16;     // 8 x 4 MFMA blocks per wave

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// One thread per 16-byte chunk; consecutive threads walk a row (reads of whole rows),
// each group of four writes the 64 bytes of one packed row.
__global__ __launch_bounds__(256) void pack_rows_kernel(const u16* __restrict__ x, int R,
                                                        int K, int64_t ldx, int64_t n_chunks,
                                                        u16* __restrict__ out) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n_chunks) return;
  const int nsteps = K / PK_K;
  const int c = int(i & 3);
  const int64_t rs = i >> 2;
  const int s = int(rs % nsteps);
  const int64_t row = rs / nsteps;
  const int r = int(row % PK_ROWS);
  const int64_t t = row / PK_ROWS;
  const uint4 v = row < R ? ld16(x + row * ldx + s * PK_K + c * 8) : make_uint4(0, 0, 0, 0);
  u16* dst = out + (t * nsteps + s) * PK_BLOCK + r * PK_K + ((c ^ ((r >> 1) & 3)) * 8);
  *reinterpret_cast<uint4*>(dst) = v;
}

// LSE epilogue in the 16x16 layout: each lane holds 32 logits of each of four entries; the
// four lane groups of an entry combine by shuffles, the two wave rows through LDS.  The
// target logit is gathered from the accumulators as in EpiLse: row r of the wave's 128 sits
// in block r / 16, element r % 4 of lane group (r / 4) % 4.
struct EpiLse16 {
  float2* partial;
  float* target;         // [N] target logits z[x_n]
  const int32_t* ids;    // [N] cached token ids
  __device__ void operator()(const f32x4 (&acc)[HMB][HNB], const GemmArgs& g, int tm, int m0w,
                             int n0w, int lane, u16* lds) const {
    const int grp = lane >> 4, c16 = lane & 15;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    float2* red = reinterpret_cast<float2*>(lds);   // [WGM][GBN] pairs
    const bool edge = tm * GBM + GBM > g.M;
    int rt[HNB];
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) rt[nb] = ids[min(n0w + nb * 16 + c16, g.N - 1)] - m0w;
    float mx[HNB], sm[HNB], mc[HNB];
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) mx[nb] = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < HMB; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = !edge || (m0w + mb * 16 + 4 * grp + e < g.M);
#pragma unroll
        for (int nb = 0; nb < HNB; ++nb)
          if (ok) mx[nb] = fmaxf(mx[nb], acc[mb][nb][e]);
      }
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) {
      mc[nb] = mx[nb] == -INFINITY ? 0.f : mx[nb] * kLog2e;
      sm[nb] = 0.f;
    }
#pragma unroll
    for (int mb = 0; mb < HMB; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = !edge || (m0w + mb * 16 + 4 * grp + e < g.M);
#pragma unroll
        for (int nb = 0; nb < HNB; ++nb)
          if (ok) sm[nb] += fast_exp2(fmaf(acc[mb][nb][e], kLog2e, -mc[nb]));
      }
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) {
      const int r = rt[nb];
      const bool own = n0w + nb * 16 + c16 < g.N && uint32_t(r) < uint32_t(GTM) &&
                       ((r >> 2) & 3) == grp;
      if (__any(own)) {
        const int idx = (r >> 4) * 4 + (r & 3);
        float z = 0.f;
#pragma unroll
        for (int mb = 0; mb < HMB; ++mb)
#pragma unroll
          for (int e = 0; e < 4; ++e) z = idx == mb * 4 + e ? acc[mb][nb][e] : z;
        if (own) target[n0w + nb * 16 + c16] = z;
      }
    }
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) {
#pragma unroll
      for (int off = 16; off < 64; off <<= 1) {
        const float mx2 = __shfl_xor(mx[nb], off);
        const float sm2 = __shfl_xor(sm[nb], off);
        const float M = fmaxf(mx[nb], mx2);
        float S = 0.f;
        if (M != -INFINITY)
          S = sm[nb] * exp2f((mx[nb] - M) * kLog2e) + sm2 * exp2f((mx2 - M) * kLog2e);
        mx[nb] = M;
        sm[nb] = S;
      }
      if (grp == 0) red[wm * GBN + wn * GTN + nb * 16 + c16] = make_float2(mx[nb], sm[nb]);
    }
    __syncthreads();
    if (wm == 0 && grp == 0) {
#pragma unroll
      for (int nb = 0; nb < HNB; ++nb) {
        const int c = wn * GTN + nb * 16 + c16;
        const int n = n0w + nb * 16 + c16;
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

__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(u >> 32));
  return reinterpret_cast<const char*>((uint64_t(hi) << 32) | lo);
}

template <int P>
using IC = std::integral_constant<int, P>;

// g.A, g.B: packed operands (M and N rows, K a multiple of 32).  Waves 0-3 stage the A block
// of a k-step, waves 4-7 the B block.  The loads are issued from inline assembly so that the
// compiler, which cannot tell the four stages apart across the loop, does not order every
// LDS read after every pending load; their completion is awaited explicitly (vmcnt) before
// the barrier that precedes the reads of each stage.
template <class Epi>
__global__ __launch_bounds__(GNT, 1) void gemm_lmhead_packed(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) u16 s0[PSTAGE];
  __shared__ __attribute__((aligned(1024))) u16 s1[PSTAGE];
  __shared__ __attribute__((aligned(1024))) u16 s2[PSTAGE];
  __shared__ __attribute__((aligned(1024))) u16 s3[PSTAGE];
  auto stg = [&](auto p) -> u16* {
    constexpr int q = decltype(p)::value % PNST;
    if constexpr (q == 0) return s0;
    else if constexpr (q == 1) return s1;
    else if constexpr (q == 2) return s2;
    else return s3;
  };
  int tm, tn;
  tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int grp = lane >> 4, r16 = lane & 15;
  const int wm = wave / WGN, wn = wave % WGN;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int nsteps = g.K / PK_K;
  const bool isA = wave_u < 4;
  const char* gbase = isA ? reinterpret_cast<const char*>(g.A + int64_t(tm) * nsteps * PK_BLOCK)
                          : reinterpret_cast<const char*>(g.B + int64_t(tn) * nsteps * PK_BLOCK);
  const uint32_t lds_w = uint32_t(wave_u * 4 * 1024);   // this wave's 4 KB of a stage
  const uint32_t goff = uint32_t(((wave_u & 3) * 4 * 64 + lane) * 16);
  // instruction j of a step: the wave's j-th 1 KB run of the block (global and LDS)
  auto dma = [&](u16* stage, int step, int j) {
    const uint64_t base = reinterpret_cast<uint64_t>(
        uniform_ptr(gbase + int64_t(min(step, nsteps - 1)) * (PK_BLOCK * 2) + j * 1024));
    const uint32_t lds = uint32_t(reinterpret_cast<uintptr_t>(stage)) + lds_w + uint32_t(j * 1024);
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(lds), "v"(goff), "s"(base) : "memory", "m0");
  };
  // fragment reads: one lane offset (row r16 of a block, chunk grp swizzled by r16 bits 1-2,
  // the same for every block); the blocks are immediate offsets
  uint32_t loff = uint32_t(r16 * 64 + ((grp ^ ((r16 >> 1) & 3)) * 16));
  const uint32_t aoff = uint32_t(wm * GTM * PK_K * 2);
  const uint32_t boff = uint32_t((GBM + wn * GTN) * PK_K * 2);
  auto fragA = [&](const u16* S, int mb) {
    return as_bf16x8(*reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + aoff +
                                                      loff + mb * 1024));
  };
  auto fragB = [&](const u16* S, int nb) {
    return as_bf16x8(*reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + boff +
                                                      loff + nb * 1024));
  };
  f32x4 acc[HMB][HNB];
#pragma unroll
  for (int mb = 0; mb < HMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < HNB; ++nb) acc[mb][nb] = f32x4{};
  bf16x8 fa[HMB], fb0[HNB], fb1[HNB];
  // s_waitcnt vmcnt(4) expcnt(7) lgkmcnt(0): this wave's loads of the next k-step have landed
  // (the following k-step's four may be in flight) and its fragment reads are complete
  constexpr int kWaitNext = 4 | (7 << 4);
  // k-step t (P = t mod 4 fixes the stages and the current B set): MFMAs of k-step t from
  // registers; fragments of k-step t+1 from its stage (A refilled block by block after the
  // block's last MFMA, B double buffered); loads of k-step t+3 into the stage that held t-1.
  auto step = [&](auto p, int t) {
    constexpr int P = decltype(p)::value;
    const bf16x8(&fbc)[HNB] = (P & 1) ? fb1 : fb0;
    bf16x8(&fbn)[HNB] = (P & 1) ? fb0 : fb1;
    const u16* Sn = stg(IC<P + 1>{});
    u16* Sd = stg(IC<P + 3>{});
    asm volatile("" : "+v"(loff));
    __builtin_amdgcn_s_waitcnt(kWaitNext);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < HMB * HNB; ++i) {
      const int mb = i / HNB, nb = i % HNB;
      acc[mb][nb] = mfma16(fa[mb], fbc[nb], acc[mb][nb]);
      if (i < HNB) fbn[i] = fragB(Sn, i);
      if (nb == HNB - 1) fa[mb] = fragA(Sn, mb);
      if ((i & 7) == 0) dma(Sd, t + 3, i >> 3);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
#pragma unroll
  for (int j = 0; j < 4; ++j) dma(s0, 0, j);
#pragma unroll
  for (int j = 0; j < 4; ++j) dma(s1, 1, j);
#pragma unroll
  for (int j = 0; j < 4; ++j) dma(s2, 2, j);
  __builtin_amdgcn_s_waitcnt(8 | (7 << 4));
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < HMB; ++mb) fa[mb] = fragA(s0, mb);
#pragma unroll
  for (int nb = 0; nb < HNB; ++nb) fb0[nb] = fragB(s0, nb);
  int t = 0;
  for (; t + PNST <= nsteps; t += PNST) {
    step(IC<0>{}, t);
    step(IC<1>{}, t + 1);
    step(IC<2>{}, t + 2);
    step(IC<3>{}, t + 3);
  }
  if (t < nsteps) step(IC<0>{}, t);
  if (t + 1 < nsteps) step(IC<1>{}, t + 1);
  if (t + 2 < nsteps) step(IC<2>{}, t + 2);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  epi(acc, g, tm, tm * GBM + wm * GTM, tn * GBN + wn * GTN, lane, s0);
}

// ------------------------------------------------------------------ FP8 path
// The same contraction on OCP E4M3 codes (one byte per element) with the gfx950
// 32x32x64 FP8 MFMA (unit block scales, so it multiplies the codes' values exactly and
// accumulates in fp32).  Rows of K bytes are moved as K/2 16-bit units: the loader, the
// LDS stages and their swizzle are those of the bf16 kernel, so one k-tile holds 128
// codes per row; a k-step of 64 codes takes 32 bytes per lane (two 16-byte chunks).
typedef int i32x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f32x16 mfma_fp8(i32x8 a, i32x8 b, f32x16 c) {
  // operand formats 0 (E4M3), block scales 127 (2^0)
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}

template <class Epi>
__global__ __launch_bounds__(GNT, 1) void gemm_tn_fp8(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) u16 lds0[STAGE];
  __shared__ __attribute__((aligned(1024))) u16 lds1[STAGE];
  int tm, tn;
  tile_of(blockIdx.x, g.tiles_m, g.tiles_n, tm, tn);
  const int m0 = tm * GBM, n0 = tn * GBN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int hi = lane >> 5, col = lane & 31;
  const int wm = wave / WGN, wn = wave % WGN;

  const u16* ga[LPW];
  const u16* gb[LPW];
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int r = (wave * LPW + j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    ga[j] = g.A + int64_t(min(m0 + r, g.M - 1)) * g.lda + c * 8;
    gb[j] = g.B + int64_t(min(n0 + r, g.N - 1)) * g.ldb + c * 8;
  }
  auto issue_half = [&](u16* stage, int k0, int h) {
    u16* base = stage + wave * LPW * 512 + h * GBM * GBK;
#pragma unroll
    for (int j = 0; j < LPW; ++j)
      __builtin_amdgcn_global_load_lds((global_void*)((h ? gb[j] : ga[j]) + k0),
                                       (lds_void*)(base + j * 512), 16, 0, 0);
  };
  // k-step ks (codes 64ks .. 64ks+63 of the tile): lane half hi takes codes 32hi .. +31,
  // i.e. 16-byte chunks 4ks + 2hi and 4ks + 2hi + 1 of its row
  auto frag = [&](const u16* S, int r, int ks) {
    const int c0 = 4 * ks + 2 * hi, sw = (r >> 1) & 7;
    const uint4 x = ld16(S + r * GBK + ((c0 ^ sw) * 8));
    const uint4 y = ld16(S + r * GBK + (((c0 + 1) ^ sw) * 8));
    return i32x8{int(x.x), int(x.y), int(x.z), int(x.w), int(y.x), int(y.y), int(y.z), int(y.w)};
  };
  f32x16 acc[GMB][GNB];
#pragma unroll
  for (int mb = 0; mb < GMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < GNB; ++nb) acc[mb][nb] = f32x16{};
  const int nk = g.K / GBK;
  // Fragments: fa holds one k-step's A fragments and is refilled block by block as soon
  // as a block's last MFMA is issued; B fragments are double buffered.  This keeps the
  // operands at 64 registers (two full sets would spill).
  i32x8 fa[GMB], fb0[GNB], fb1[GNB];
  auto rowA = [&](int mb) { return wm * GTM + mb * 32 + col; };
  auto rowB = [&](int nb) { return GBM + wn * GTN + nb * 32 + col; };
  // One k-step: MFMAs on (fa, fbc); the next k-step's fragments come from stage Sn at
  // k-step ksn; `dma` issues this step's direct loads, one after every other MFMA.
  auto kstep = [&](const i32x8 (&fbc)[GNB], i32x8 (&fbn)[GNB], const u16* Sn, int ksn,
                   auto dma) {
#pragma unroll
    for (int i = 0; i < GMB * GNB; ++i) {
      const int mb = i / GNB, nb = i % GNB;
      acc[mb][nb] = mfma_fp8(fa[mb], fbc[nb], acc[mb][nb]);
      if (i < GNB) fbn[i] = frag(Sn, rowB(i), ksn);
      if (nb == GNB - 1) fa[mb] = frag(Sn, rowA(mb), ksn);
      if ((i & 1) == 0) dma(i >> 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto no_dma = [](int) {};
  // one k-tile from `cur`: k-step 0 carries the B half of `nxt` (k-tile kt+1); after the
  // barrier that frees `cur`, k-step 1 refills its A half with k-tile kt+2
  auto tile = [&](const u16* cur, u16* nxt, int kt) {
    __builtin_amdgcn_sched_barrier(0);
    const int kb = min(kt + 1, nk - 1) * GBK, ka = min(kt + 2, nk - 1) * GBK;
    u16* bdst = nxt + wave * LPW * 512 + GBM * GBK;
    kstep(fb0, fb1, cur, 1, [&](int j) {
      __builtin_amdgcn_global_load_lds((global_void*)(gb[j] + kb), (lds_void*)(bdst + j * 512),
                                       16, 0, 0);
    });
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    u16* adst = const_cast<u16*>(cur) + wave * LPW * 512;
    kstep(fb1, fb0, nxt, 0, [&](int j) {
      __builtin_amdgcn_global_load_lds((global_void*)(ga[j] + ka), (lds_void*)(adst + j * 512),
                                       16, 0, 0);
    });
  };
  (void)no_dma;
  issue_half(lds0, 0, 0);
  issue_half(lds0, 0, 1);
  issue_half(lds1, min(1, nk - 1) * GBK, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < GMB; ++mb) fa[mb] = frag(lds0, rowA(mb), 0);
#pragma unroll
  for (int nb = 0; nb < GNB; ++nb) fb0[nb] = frag(lds0, rowB(nb), 0);
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    tile(lds0, lds1, kt);
    tile(lds1, lds0, kt + 1);
  }
  if (kt < nk) tile(lds0, lds1, kt);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  epi(acc, g, tm, m0 + wm * GTM, n0 + wn * GTN, lane, lds0);
}

// E4M3 quantization: amax = max |x| over a row (or the matrix), codes = E4M3(x * (448 /
// amax)) rounded to nearest even by the conversion instruction, scale = amax / 448 (fp32
// throughout; an all-zero row gives codes 0 and scale 0).  Rows are read four elements
// per load (8 bytes of bf16 or 16 bytes of fp32; cols is a multiple of 4).
struct Quad {
  float v[4];
};
template <class T>
__device__ __forceinline__ Quad ld4(const T* p);
template <>
__device__ __forceinline__ Quad ld4<u16>(const u16* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return Quad{{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
               __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u)}};
}
template <>
__device__ __forceinline__ Quad ld4<float>(const float* p) {
  const float4 f = *reinterpret_cast<const float4*>(p);
  return Quad{{f.x, f.y, f.z, f.w}};
}

__device__ __forceinline__ float block_max_256(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  v = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  return v;
}

template <class T>
__device__ __forceinline__ float row_amax(const T* row, int cols, float* red) {
  float m = 0.f;
  for (int c = threadIdx.x * 4; c < cols; c += 1024) {
    const Quad q = ld4<T>(row + c);
    m = fmaxf(m, fmaxf(fmaxf(fabsf(q.v[0]), fabsf(q.v[1])), fmaxf(fabsf(q.v[2]), fabsf(q.v[3]))));
  }
  return block_max_256(m, red);
}

template <class T>
__device__ __forceinline__ void quantize_row(const T* row, int cols, float amax, uint8_t* q) {
  const float inv = amax > 0.f ? 448.f / amax : 0.f;
  uint32_t* out = reinterpret_cast<uint32_t*>(q);
  for (int c = threadIdx.x * 4; c < cols; c += 1024) {
    const Quad x = ld4<T>(row + c);
    int v = __builtin_amdgcn_cvt_pk_fp8_f32(x.v[0] * inv, x.v[1] * inv, 0, false);
    v = __builtin_amdgcn_cvt_pk_fp8_f32(x.v[2] * inv, x.v[3] * inv, v, true);
    out[c >> 2] = uint32_t(v);
  }
}

// one scale per row: a workgroup per row reads it twice (the second pass hits the cache)
template <class T>
__global__ __launch_bounds__(256) void quantize_rows_kernel(const T* __restrict__ x, int cols,
                                                            uint8_t* __restrict__ q,
                                                            float* __restrict__ scale) {
  __shared__ float red[4];
  const int64_t r = blockIdx.x;
  const float amax = row_amax<T>(x + r * cols, cols, red);
  if (threadIdx.x == 0) scale[r] = amax / 448.f;
  quantize_row<T>(x + r * cols, cols, amax, q + r * cols);
}

// one scale for the matrix: row maxima, their maximum, then the codes
template <class T>
__global__ __launch_bounds__(256) void row_amax_kernel(const T* __restrict__ x, int cols,
                                                       float* __restrict__ amax) {
  __shared__ float red[4];
  const float m = row_amax<T>(x + int64_t(blockIdx.x) * cols, cols, red);
  if (threadIdx.x == 0) amax[blockIdx.x] = m;
}

__global__ __launch_bounds__(1024) void max_reduce_kernel(const float* __restrict__ v, int64_t n,
                                                          float* __restrict__ out) {
  __shared__ float red[16];
  float m = 0.f;
  for (int64_t i = threadIdx.x; i < n; i += 1024) m = fmaxf(m, v[i]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = red[0];
    for (int w = 1; w < 16; ++w) t = fmaxf(t, red[w]);
    out[0] = t;
  }
}

template <class T>
__global__ __launch_bounds__(256) void quantize_matrix_kernel(const T* __restrict__ x, int cols,
                                                              const float* __restrict__ amax,
                                                              uint8_t* __restrict__ q,
                                                              float* __restrict__ scale) {
  const int64_t r = blockIdx.x;
  if (r == 0 && threadIdx.x == 0) scale[0] = amax[0] / 448.f;
  quantize_row<T>(x + r * cols, cols, amax[0], q + r * cols);
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
// gi, gi+64, ... of entry e (16 consecutive entries read 128 contiguous bytes of a tile's
// row of partials; up to 512 tiles are eight loads per thread, all in flight at once), then
// the 64 groups are folded by shuffles within each wave and across the waves in LDS.
constexpr int CMB_E = 16, CMB_G = 64;

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
  __shared__ float2 red[CMB_E * CMB_G / 64][CMB_E];
  const int e = threadIdx.x % CMB_E, gi = threadIdx.x / CMB_E;
  const int n = blockIdx.x * CMB_E + e;
  float M = -INFINITY, S = 0.f;
  if (n < N) {
    // eight independent loads in flight per thread (tiles past the end fold as empty)
    for (int t0 = gi; t0 < n_tiles; t0 += 8 * CMB_G) {
      float2 p[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int t = t0 + q * CMB_G;
        p[q] = t < n_tiles ? partial[int64_t(t) * N + n] : make_float2(-INFINITY, 0.f);
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) lse_fold(M, S, p[q].x, p[q].y);
    }
  }
  // the four groups of an entry within a wave (lanes e, e+16, e+32, e+48) fold by
  // shuffles, then the waves' results through LDS
#pragma unroll
  for (int off = 16; off < 64; off <<= 1) {
    const float m2 = __shfl_xor(M, off), s2 = __shfl_xor(S, off);
    lse_fold(M, S, m2, s2);
  }
  constexpr int NWV = CMB_E * CMB_G / 64;
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) < CMB_E) red[wv][e] = make_float2(M, S);
  __syncthreads();
  if (gi == 0 && n < N) {
    float Mt = -INFINITY, St = 0.f;
#pragma unroll
    for (int r = 0; r < NWV; ++r) lse_fold(Mt, St, red[r][e].x, red[r][e].y);
    const float lse = Mt + logf(St);
    // sequence of entry n: the last b with cu[b] <= n
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= n) lo = mid; else hi = mid - 1;
    }
    const bool last = n == cu[lo + 1] - 1;
    const bool frozen = n - cu[lo] < n_frozen;
    // -log P >= 0: for a near-certain token (z[x_n] the row maximum, every other term
    // tiny) rounding in the exponentials and the logarithm can take the difference a few
    // ulps below zero; it is clamped there (a NaN stays NaN)
    const float d = lse - target[n];
    scores[n] = (last || frozen) ? INFINITY : (d < 0.f ? 0.f : d);
    if (lse_out) lse_out[n] = lse;
  }
}

// out[c][r] = in[r][c] for an in [rows][cols] matrix: 64x64 tiles through LDS (one
// padding column, so the column reads hit distinct banks).  Used once per model to lay
// W_o out K-contiguous for the fused LM-head weight.
template <class T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, T* __restrict__ out,
                                                        int rows, int cols) {
  __shared__ T tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = in[int64_t(r) * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) out[int64_t(c) * rows + r] = tile[tx][i];
  }
}

}  // namespace

hipError_t launch_transpose(int dtype, const void* in, void* out, int rows, int cols,
                            hipStream_t s) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  if (dtype == CC_BF16)
    hipLaunchKernelGGL(transpose_kernel<u16>, grid, dim3(256), 0, s, static_cast<const u16*>(in),
                       static_cast<u16*>(out), rows, cols);
  else
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s,
                       static_cast<const float*>(in), static_cast<float*>(out), rows, cols);
  return hipGetLastError();
}

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

size_t packed_rows_bytes(int64_t rows, int cols) {
  return size_t((rows + PK_ROWS - 1) / PK_ROWS) * PK_ROWS * size_t(cols) * 2;
}

hipError_t launch_pack_rows(const void* x, int64_t rows, int cols, int64_t ldx, void* out,
                            hipStream_t s) {
  const int64_t tiles = (rows + PK_ROWS - 1) / PK_ROWS;
  const int64_t n_chunks = tiles * PK_ROWS * (cols / PK_K) * 4;
  if (n_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_rows_kernel, dim3(unsigned((n_chunks + 255) / 256)), dim3(256), 0, s,
                     static_cast<const u16*>(x), int(rows), cols, ldx, n_chunks,
                     static_cast<u16*>(out));
  return hipGetLastError();
}

hipError_t launch_lmhead(const LmHeadLaunch& a, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  int n_vt;
  if (a.dtype == CC_BF16 && a.w_packed != nullptr) {
    hipError_t err = launch_pack_rows(a.u, a.N, a.D, a.D, a.u_packed, s);
    if (err != hipSuccess) return err;
    GemmArgs g;
    g.A2 = nullptr;
    g.A = static_cast<const u16*>(a.w_packed);
    g.B = static_cast<const u16*>(a.u_packed);
    g.M = a.V;
    g.N = a.N;
    g.K = a.D;
    g.lda = g.ldb = 0;   // unused: packed operands
    g.tiles_n = (a.N + GBN - 1) / GBN;
    n_vt = (a.V + GBM - 1) / GBM;
    g.tiles_m = n_vt;
    EpiLse16 e{a.partial, a.target, a.ids};
    hipLaunchKernelGGL(gemm_lmhead_packed<EpiLse16>, dim3(n_vt * g.tiles_n), dim3(GNT), 0, s, g, e);
  } else if (a.dtype == CC_BF16) {
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

hipError_t launch_quantize_e4m3(int dtype, const void* x, int64_t rows, int cols, int per_row,
                                uint8_t* q, float* scale, float* amax_ws, hipStream_t s) {
  if (rows == 0 || cols == 0) return hipSuccess;
  const bool bf = dtype == CC_BF16;
  if (per_row) {
    if (bf)
      hipLaunchKernelGGL(quantize_rows_kernel<u16>, dim3(rows), dim3(256), 0, s,
                         static_cast<const u16*>(x), cols, q, scale);
    else
      hipLaunchKernelGGL(quantize_rows_kernel<float>, dim3(rows), dim3(256), 0, s,
                         static_cast<const float*>(x), cols, q, scale);
    return hipGetLastError();
  }
  if (bf)
    hipLaunchKernelGGL(row_amax_kernel<u16>, dim3(rows), dim3(256), 0, s,
                       static_cast<const u16*>(x), cols, amax_ws);
  else
    hipLaunchKernelGGL(row_amax_kernel<float>, dim3(rows), dim3(256), 0, s,
                       static_cast<const float*>(x), cols, amax_ws);
  hipLaunchKernelGGL(max_reduce_kernel, dim3(1), dim3(1024), 0, s, amax_ws, rows, amax_ws + rows);
  if (bf)
    hipLaunchKernelGGL(quantize_matrix_kernel<u16>, dim3(rows), dim3(256), 0, s,
                       static_cast<const u16*>(x), cols, amax_ws + rows, q, scale);
  else
    hipLaunchKernelGGL(quantize_matrix_kernel<float>, dim3(rows), dim3(256), 0, s,
                       static_cast<const float*>(x), cols, amax_ws + rows, q, scale);
  return hipGetLastError();
}

hipError_t launch_lmhead_fp8(const LmHeadFp8Launch& a, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  hipError_t err = launch_quantize_e4m3(a.dtype, a.u, a.N, a.D, 1, a.uq, a.su, a.amax_ws, s);
  if (err != hipSuccess) return err;
  GemmArgs g;
  g.A2 = nullptr;
  g.A = reinterpret_cast<const u16*>(a.wq);   // rows of D codes = D/2 16-bit units
  g.B = reinterpret_cast<const u16*>(a.uq);
  g.M = a.V;
  g.N = a.N;
  g.K = a.D / 2;
  g.lda = a.D / 2;
  g.ldb = a.D / 2;
  g.tiles_n = (a.N + GBN - 1) / GBN;
  const int n_vt = (a.V + GBM - 1) / GBM;
  g.tiles_m = n_vt;
  EpiLse e{a.partial, a.target, a.ids, a.su, a.sw};
  hipLaunchKernelGGL(gemm_tn_fp8<EpiLse>, dim3(n_vt * g.tiles_n), dim3(GNT), 0, s, g, e);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  hipLaunchKernelGGL(lse_combine, dim3((a.N + CMB_E - 1) / CMB_E), dim3(CMB_E * CMB_G), 0, s,
                     a.partial, n_vt, a.target, a.cu_d, a.n_seqs, a.n_frozen, a.N, a.scores,
                     a.lse);
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

int gemm_split_slices(int M, int N, int K) {
  const int tiles = ((M + GBM - 1) / GBM) * ((N + GBN - 1) / GBN);
  const int nk = K / GBK;
  if (tiles >= 128 || nk < 8) return 1;
  // up to one workgroup per CU, at least four k-tiles per slice, at most 5 slices: more
  // slices add partial sums to write and reduce faster than they add parallelism (measured at
  // 42 tiles, 768 entries: 3, 4, 5 and 7 slices give 1.28, 1.26, 1.25 and 1.31 ms per refresh)
  const int want = std::max(1, std::min({(256 + tiles - 1) / tiles, nk / 4, 5}));
  const int per = (nk + want - 1) / want;
  return (nk + per - 1) / per;
}

namespace {
// k-tiles per slice for the slice count gemm_split_slices chose
int split_ktiles(int K, int S) {
  const int nk = K / GBK;
  return (nk + S - 1) / S;
}
}  // namespace

hipError_t launch_qproj_rope(const void* wq, const void* a, void* q, const float2* rot, int N,
                             int D, int HD, float* part, hipStream_t s) {
  if (N == 0) return hipSuccess;
  GemmArgs g = make_args(wq, a, HD, N, D, D, D);
  const int S = gemm_split_slices(HD, N, D);
  if (S > 1) {
    g.kt_split = split_ktiles(D, S);
    EpiPartial<true> e{part};
    hipLaunchKernelGGL(gemm_tn_bf16<EpiPartial<true>>, dim3(g.tiles_m * g.tiles_n, S), dim3(GNT),
                       0, s, g, e);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int64_t threads = int64_t(N) * (HD / 2);
    hipLaunchKernelGGL(reduce_rope, dim3(unsigned((threads + 255) / 256)), dim3(256), 0, s, part,
                       S, N, HD, rot, static_cast<u16*>(q));
    return hipGetLastError();
  }
  EpiRope e{static_cast<u16*>(q), rot};
  hipLaunchKernelGGL(gemm_tn_bf16<EpiRope>, dim3(g.tiles_m * g.tiles_n), dim3(GNT), 0, s, g, e);
  return hipGetLastError();
}

hipError_t launch_linear_residual(const void* x, const void* w, float* h, int M, int N, int K,
                                  float* part, hipStream_t s) {
  if (M == 0) return hipSuccess;
  GemmArgs g = make_args(x, w, M, N, K, K, K);
  const int S = gemm_split_slices(M, N, K);
  if (S > 1) {
    g.kt_split = split_ktiles(K, S);
    EpiPartial<false> e{part};
    hipLaunchKernelGGL(gemm_tn_bf16<EpiPartial<false>>, dim3(g.tiles_m * g.tiles_n, S),
                       dim3(GNT), 0, s, g, e);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    const int64_t count = int64_t(M) * N;
    hipLaunchKernelGGL(reduce_residual, dim3(unsigned((count / 4 + 255) / 256)), dim3(256), 0, s,
                       part, S, count, h);
    return hipGetLastError();
  }
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
