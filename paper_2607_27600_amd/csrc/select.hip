// Keep selection of the memory-refresh cycle (Sec. 3.2): per segment, the k entries that
// come first under (score descending, ties to the lower index), emitted in ascending
// index order so the compacted cache keeps the original time order.
//
// One workgroup per segment at a time.  Scores map to order-preserving 32-bit keys (-0 ==
// +0, NaN below -inf).  8-bit radix passes over the keys (LDS histograms, wave-parallel bucket
// search) find the k-th largest key T and how many entries equal to T are kept; a final
// pass in index order emits every key > T and the lowest-index ties with block-wide
// ballot/prefix counts.  Integer work only: the result is exact.  Launches whose longest
// segment holds 8193..32768 scores keep every segment in registers (one read of the
// scores); the others re-read the scores from memory at every pass.
#include <algorithm>

#include "cc_internal.h"

namespace cc {
namespace {

constexpr int SNT = 1024;           // threads per segment
constexpr int SWAVES = SNT / 64;

// Descriptor of segment b: computed for regular launches, else by value in the kernel
// arguments (the first SEL_INLINE) or from the uploaded table.
__device__ __forceinline__ SelSeg seg_desc(const SelInline& inl, const SelSeg* segs, int b) {
  if (inl.regular)
    return SelSeg{inl.start0 + int64_t(b) * inl.stride, inl.len, inl.k, int64_t(b) * inl.k};
  return b < inl.n ? inl.s[b] : segs[b];
}

// Wave-wide inclusive scans and reductions on DPP lane moves (VALU only, no LDS round
// trip): shifts of 1, 2, 4 and 8 lanes inside each row of 16 (lanes without a source keep
// the identity), then the last lane of row 0 (2) added into row 1 (3), then lane 31 into
// rows 2 and 3.  Lane i ends with op over lanes 0..i.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x, uint32_t identity) {
  return uint32_t(__builtin_amdgcn_update_dpp(int(identity), int(x), CTRL, ROWS, 0xf, false));
}
template <class Op>
__device__ __forceinline__ uint32_t wave_scan(uint32_t x, uint32_t identity, Op op) {
  x = op(x, dpp_move<0x111, 0xf>(x, identity));   // row_shr:1
  x = op(x, dpp_move<0x112, 0xf>(x, identity));   // row_shr:2
  x = op(x, dpp_move<0x114, 0xf>(x, identity));   // row_shr:4
  x = op(x, dpp_move<0x118, 0xf>(x, identity));   // row_shr:8
  x = op(x, dpp_move<0x142, 0xa>(x, identity));   // row_bcast:15 into rows 1 and 3
  x = op(x, dpp_move<0x143, 0xc>(x, identity));   // row_bcast:31 into rows 2 and 3
  return x;
}
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x, int lane) {
  (void)lane;
  return wave_scan(x, 0u, [](uint32_t a, uint32_t b) { return a + b; });
}
// the reduction over the whole wave, in every lane
template <class Op>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t x, uint32_t identity, Op op) {
  return uint32_t(__builtin_amdgcn_readlane(int(wave_scan(x, identity, op)), 63));
}

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;   // NaN: lowest
  if ((u & 0x7fffffffu) == 0u) u = 0u;              // -0 == +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix count of `flag` over the workgroup (in thread order) and the total.
__device__ __forceinline__ int block_scan(bool flag, int* wsum, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t bal = __ballot(flag);
  const int below = __popcll(bal & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wave] = __popcll(bal);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < SWAVES; ++w) {
    const int c = wsum[w];
    before += w < wave ? c : 0;
    tot += c;
  }
  __syncthreads();
  total = tot;
  return before + below;
}

__global__ __launch_bounds__(SNT) void select_keep_kernel(const float* __restrict__ scores,
                                                          const SelSeg* __restrict__ segs,
                                                          SelInline inl,
                                                          int32_t* __restrict__ keep) {
  __shared__ uint32_t hist[256];
  __shared__ int wsum[SWAVES];
  __shared__ uint32_t sh_digit, sh_rem, sh_cnt;
  const SelSeg sg = seg_desc(inl, segs, int(blockIdx.x));
  const float* s = scores + sg.start;
  int32_t* out = keep + sg.out;
  const int n = sg.len, k = sg.k;
  const int tid = threadIdx.x;
  if (k <= 0) return;
  if (k >= n) {
    for (int i = tid; i < n; i += SNT) out[i] = i;
    return;
  }

  uint32_t prefix = 0u, mask = 0u, rem = uint32_t(k);
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < 256; i += SNT) hist[i] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += SNT) {
      const uint32_t key = order_key(s[i]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending); find the bucket holding the
      // rem-th largest candidate.
      const int lane = tid;
      uint32_t c[4], sum = 0u;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        c[j] = hist[255 - 4 * lane - j];
        sum += c[j];
      }
      const uint32_t incl = wave_incl_scan(sum, lane);   // over lanes (descending digits)
      const uint32_t excl = incl - sum;
      if (excl < rem && incl >= rem) {
        uint32_t acc = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (acc + c[j] >= rem) {
            sh_digit = uint32_t(255 - 4 * lane - j);
            sh_rem = rem - acc;
            sh_cnt = c[j];
            break;
          }
          acc += c[j];
        }
      }
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    rem = sh_rem;
    __syncthreads();
  }
  const uint32_t T = prefix;   // the k-th largest key; keep `rem` of the entries equal to T
  // the last pass's bucket holds exactly the keys equal to T: when all of them are kept,
  // ties need no ranking
  const bool all_ties = sh_cnt == rem;

  int ties_before = 0, emitted = 0;
  for (int base = 0; base < n; base += SNT) {
    const int i = base + tid;
    const uint32_t key = i < n ? order_key(s[i]) : 0u;
    const bool eq = i < n && key == T;
    const bool gt = i < n && key > T;
    int eq_total = 0, tie_rank = 0;
    if (!all_ties) tie_rank = ties_before + block_scan(eq, wsum, eq_total);
    const bool take = gt || (eq && (all_ties || uint32_t(tie_rank) < rem));
    int take_total;
    const int pos = emitted + block_scan(take, wsum, take_total);
    if (take) out[pos] = i;
    ties_before += eq_total;
    emitted += take_total;
  }
}

// ------------------------------------------------------------------ register path
// Segments of up to RMAX scores: the workgroup reads its segment once into registers and
// never touches it again.  The segment is cut into 8 chunks of 4096 scores; thread t of
// 1024 holds scores 4t .. 4t+3 of every chunk (one 16-byte load per chunk, 1 KB per wave
// instruction), so index order is (chunk, thread, slot).  The kernel is bound by vector ALU
// issue, so every per-key step is kept to a few instructions:
//  - Keys: the float's sign and magnitude turned into a signed two's complement integer
//    (-0 and +0 both become 0).  NaN keys then lie outside the keys of -inf .. +inf; a
//    segment that holds any (seen in its extremes) sets them all to one key below -inf.
//  - Extremes: the smallest key kmin and the largest key other than +inf (a max over
//    key + 2^23, where +inf alone wraps to the bottom).  The radix digits run on
//    rel = min(key - kmin, rcap), rcap = that largest key - kmin + 1: +inf keys become rcap,
//    one above every finite key, and the first digit spreads over the finite scores'
//    actual range (the +inf of a sequence's last entry would otherwise squeeze them all
//    into one bucket).
//  - One 11-bit pass over every key (no test: the first digit holds the top bits of every
//    rel) into a 2048-bin LDS histogram.  An 11-bit digit leaves about an eighth of the keys
//    an 8-bit one would in the bucket that holds the threshold, and spreads a wave's atomics
//    over more bins, so fewer lanes of one instruction collide.  When that bucket has at
//    most CMAX keys, they copy their low bits to LDS (positions from one LDS counter) and
//    one wave finishes the lower digits on that list (9 bits a pass, no block-wide
//    barrier); otherwise further 11-bit block-wide passes run over the registers.
//  - Bucket searches are two-level wave scans: lane sums over the lanes' bin ranges, then
//    the bins of the lane that holds the rank.
//  - Emission: a thread's flagged keys per chunk are counted, and one batched scan over
//    the workgroup (8 chunk counts per thread, two per word) gives every flagged key its
//    rank in index order: first for the ties (when not all of them are kept), then for
//    the kept keys, which each thread stores at their ranks (consecutive keys of a chunk
//    at consecutive ranks) through a buffer descriptor bounded by the segment's budget.
constexpr int RNT = 1024;
constexpr int RWAVES = RNT / 64;
constexpr int RCW = 4;                 // scores per thread per chunk
constexpr int RCH = 8;                 // chunks
constexpr int RCHUNK = RNT * RCW;      // scores per chunk
constexpr int RPT = RCH * RCW;         // scores per thread
constexpr int RMAX = RNT * RPT;
constexpr int CMAX = 4096;             // candidate list of the one-wave finish
constexpr int SD = 11;                 // bits of a block-wide digit
constexpr int SBINS = 1 << SD;
constexpr int WD = 9;                  // bits of a digit of the one-wave finish
constexpr int WBINS = 1 << WD;
constexpr int32_t KEY_PINF = 0x7f800000;    // key of +inf
constexpr int32_t KEY_NINF = -0x7f800000;   // key of -inf
constexpr int32_t KEY_NAN = KEY_NINF - 1;   // key of every NaN
constexpr uint32_t FIN_SHIFT = 0x00800000u; // key + FIN_SHIFT wraps +inf, and only +inf, to INT_MIN
constexpr int32_t I32_MAX = 0x7fffffff;
constexpr int32_t I32_MIN = -I32_MAX - 1;

// Signed order key of a float's bits: sign and magnitude to two's complement.
__device__ __forceinline__ int32_t skey(uint32_t u) {
  const uint32_t t = uint32_t(int32_t(u) >> 31);
  return int32_t((u ^ t) + (t & 0x80000001u));
}

// Inclusive scan inside each row of 16 lanes (row 0 holds lanes 0..15).
__device__ __forceinline__ uint32_t row_scan(uint32_t x) {
  x += dpp_move<0x111, 0xf>(x, 0u);
  x += dpp_move<0x112, 0xf>(x, 0u);
  x += dpp_move<0x114, 0xf>(x, 0u);
  x += dpp_move<0x118, 0xf>(x, 0u);
  return x;
}
// op over lanes 0..15, in every lane
template <class Op>
__device__ __forceinline__ uint32_t row0_reduce(uint32_t x, uint32_t identity, Op op) {
  x = op(x, dpp_move<0x111, 0xf>(x, identity));
  x = op(x, dpp_move<0x112, 0xf>(x, identity));
  x = op(x, dpp_move<0x114, 0xf>(x, identity));
  x = op(x, dpp_move<0x118, 0xf>(x, identity));
  return uint32_t(__builtin_amdgcn_readlane(int(x), 15));
}
constexpr auto imin = [](uint32_t a, uint32_t b) { return uint32_t(min(int32_t(a), int32_t(b))); };
constexpr auto imax = [](uint32_t a, uint32_t b) { return uint32_t(max(int32_t(a), int32_t(b))); };

struct Pick {
  uint32_t digit, rem, cnt;
};

// Run by one whole wave: in a histogram of 64 * BPL bins searched from the highest bin down,
// the bin holding the rem-th largest counted key (1 <= rem <= total), the rank left inside
// it and its count; every lane receives the result.  Level 1: lane l sums bins
// 64 BPL - BPL (l + 1) .. 64 BPL - 1 - BPL l and a wave scan finds the lane whose range
// holds the rank; level 2: lane j < BPL reads that range's j-th highest bin and a second
// scan finds the bin.
template <int BPL>
__device__ __forceinline__ Pick pick_bucket(const uint32_t* h, uint32_t rem, int lane) {
  constexpr int NB = 64 * BPL;
  const uint32_t* mine = h + NB - BPL * (lane + 1);
  uint32_t sum = 0u;
  if constexpr (BPL % 4 == 0) {
#pragma unroll
    for (int q = 0; q < BPL / 4; ++q) {
      const uint4 v = reinterpret_cast<const uint4*>(mine)[q];
      sum += (v.x + v.y) + (v.z + v.w);
    }
  } else {
#pragma unroll
    for (int q = 0; q < BPL; ++q) sum += mine[q];
  }
  const uint32_t incl = wave_incl_scan(sum, lane);
  const uint64_t over = __ballot(incl >= rem);
  const int owner = over ? int(__builtin_ctzll(over)) : 63;   // rem <= total: some lane does
  const uint32_t before = uint32_t(__builtin_amdgcn_readlane(int(incl - sum), owner));
  const int top = NB - BPL * owner - 1;              // the owner's highest bin
  const uint32_t c = lane < BPL ? h[top - lane] : 0u;
  const uint32_t incl2 = wave_incl_scan(c, lane);
  const uint64_t hit = __ballot(lane < BPL && before + incl2 >= rem);
  const int j = hit ? int(__builtin_ctzll(hit)) : BPL - 1;
  const uint32_t cj = uint32_t(__builtin_amdgcn_readlane(int(c), j));
  const uint32_t ij = uint32_t(__builtin_amdgcn_readlane(int(incl2), j));
  return {uint32_t(top - j), rem - before - (ij - cj), cj};
}

// Ranks in index order of flagged keys: base[c] = flagged keys before this thread's part of
// chunk c.  wtot: [RWAVES][RCH / 2] words of
// LDS owned by this call (16-byte aligned rows); wave: the wave's index, uniform.  Contains
// one barrier.  After it, lanes 0..15 of every wave scan the 16 waves' totals.
static_assert(RPT == 32, "one bit per key in a 32-bit mask");
static_assert(RWAVES == 16, "the waves' totals are combined in one row of 16 lanes");
// own[q]: this thread's flagged keys in chunks 2q (low half) and 2q + 1 (high half).
__device__ __forceinline__ void chunk_offsets(const uint32_t (&own)[RCH / 2], uint32_t (&base)[RCH],
                                              uint32_t (*wtot)[RCH / 2], int lane, int wave) {
  uint32_t inc[RCH / 2];
#pragma unroll
  for (int q = 0; q < RCH / 2; ++q) {
    // inclusive scan over the wave, two chunks per word (a field stays below 4 * 64 + 1)
    inc[q] = wave_incl_scan(own[q], lane);
  }
  if (lane == 63) *reinterpret_cast<uint4*>(wtot[wave]) = make_uint4(inc[0], inc[1], inc[2], inc[3]);
  __syncthreads();
  uint4 t = make_uint4(0u, 0u, 0u, 0u);
  if (lane < RWAVES) t = *reinterpret_cast<const uint4*>(wtot[lane]);
  const uint32_t tv[4] = {t.x, t.y, t.z, t.w};
  uint32_t run = 0u;
#pragma unroll
  for (int q = 0; q < RCH / 2; ++q) {
    const uint32_t sc = row_scan(tv[q]);
    const uint32_t all = uint32_t(__builtin_amdgcn_readlane(int(sc), RWAVES - 1));
    const uint32_t bef = uint32_t(__builtin_amdgcn_readlane(int(sc - tv[q]), wave));
    const uint32_t mine = bef + inc[q] - own[q];
    base[2 * q] = run + (mine & 0xffffu);
    run += all & 0xffffu;
    base[2 * q + 1] = run + (mine >> 16);
    run += all >> 16;
  }
}

// own[] of chunk_offsets from a mask (bit 4c + i: slot i of chunk c)
__device__ __forceinline__ void chunk_counts(uint32_t m, uint32_t (&own)[RCH / 2]) {
#pragma unroll
  for (int q = 0; q < RCH / 2; ++q)
    own[q] = uint32_t(__popc((m >> (8 * q)) & 0xfu)) | (uint32_t(__popc((m >> (8 * q + 4)) & 0xfu)) << 16);
}

struct RegLds {
  uint32_t hist[SBINS];
  uint32_t cand[CMAX];
  uint32_t whist[WBINS];
  uint32_t red[5][RWAVES];
  __attribute__((aligned(16))) uint32_t wtot[2][RWAVES][RCH / 2];
  uint32_t sh_digit, sh_rem, sh_cnt, sh_ncand;
};

// The descriptor's fields in scalar registers (a descriptor picked from the kernel
// arguments by the block index is otherwise not known to be uniform).
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(uint64_t(x)))));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readfirstlane(int(uint32_t(uint64_t(x) >> 32))));
  return int64_t((uint64_t(hi) << 32) | lo);
}

__global__ __launch_bounds__(RNT, 1) void select_keep_regs(const float* __restrict__ scores,
                                                           const SelSeg* __restrict__ segs,
                                                           SelInline inl, int n_segs,
                                                           int32_t* __restrict__ keep) {
  __shared__ __attribute__((aligned(16))) RegLds L;
  // Workgroups walk the segments (one per CU; the kernel's registers allow no second):
  // the stores of one segment drain while the loads of the next are in flight.
  for (int sgi = blockIdx.x; sgi < n_segs; sgi += gridDim.x) {
    // thread indices opaque per iteration: nothing derived from them is hoisted out of the loop
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    SelSeg sg = seg_desc(inl, segs, sgi);
    sg.start = uniform64(sg.start);
    sg.out = uniform64(sg.out);
    sg.len = __builtin_amdgcn_readfirstlane(sg.len);
    sg.k = __builtin_amdgcn_readfirstlane(sg.k);
    const int n = sg.len, k = sg.k;
    int32_t* out = keep + sg.out;
    if (k <= 0) continue;
    if (k >= n) {
      for (int i = tid; i < n; i += RNT) out[i] = i;
      continue;
    }
    // key[4c + i] = score c * RCHUNK + 4 * tid + i, read from a uniform base plus a 32-bit
    // byte offset.  With a 16-byte aligned start and a length divisible by four, one 16-byte
    // load per chunk (chunks past the end re-read the last four scores); otherwise four
    // loads per chunk (indices past the end re-read the last score).  Keys past the end are
    // marked padding below.
    const char* sb = reinterpret_cast<const char*>(scores + sg.start);
    uint32_t key[RPT];
    int t4 = 4 * tid;
    if ((reinterpret_cast<uintptr_t>(sb) & 15u) == 0u && (n & 3) == 0) {
#pragma unroll
      for (int c = 0; c < RCH; ++c) {
        const uint32_t off = uint32_t(min(c * RCHUNK + t4, n - 4)) * 4u;
        const uint4 v = *reinterpret_cast<const uint4*>(sb + off);
        key[4 * c] = v.x;
        key[4 * c + 1] = v.y;
        key[4 * c + 2] = v.z;
        key[4 * c + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        const uint32_t off = uint32_t(min((j >> 2) * RCHUNK + t4 + (j & 3), n - 1)) * 4u;
        key[j] = *reinterpret_cast<const uint32_t*>(sb + off);
      }
    }
    // Index arithmetic restarts from an opaque copy of 4*tid here and before the stores, so
    // the compiler recomputes it instead of keeping 64 indices (and their compare masks)
    // live across the kernel.  vbits: bit j set when key j lies inside the segment.
    asm volatile("" : "+v"(t4));
    uint32_t vbits = 0u;
#pragma unroll
    for (int c = 0; c < RCH; ++c) {
      // slots i < n - (c * RCHUNK + 4 tid) of chunk c hold scores
      const int nv = min(max(n - c * RCHUNK - t4, 0), RCW);
      vbits |= ((1u << nv) - 1u) << (RCW * c);
    }
    const bool whole = vbits == 0xffffffffu;   // every key of this thread lies inside the segment
    auto valid = [&](int j) { return ((vbits >> j) & 1u) != 0u; };

    // keys; their smallest, their largest (NaN detection) and the largest + FIN_SHIFT
    int32_t mn = I32_MAX, mx = I32_MIN, mf = I32_MIN;
    if (whole) {
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        const int32_t s = skey(key[j]);
        key[j] = uint32_t(s);
        mn = min(mn, s);
        mx = max(mx, s);
        mf = max(mf, int32_t(uint32_t(s) + FIN_SHIFT));
      }
    } else {
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        const int32_t s = skey(key[j]);
        key[j] = uint32_t(s);
        const bool v = valid(j);
        mn = v ? min(mn, s) : mn;
        mx = v ? max(mx, s) : mx;
        mf = v ? max(mf, int32_t(uint32_t(s) + FIN_SHIFT)) : mf;
      }
    }
    {
      const uint32_t r0 = wave_reduce(uint32_t(mn), uint32_t(I32_MAX), imin);
      const uint32_t r1 = wave_reduce(uint32_t(mx), uint32_t(I32_MIN), imax);
      const uint32_t r2 = wave_reduce(uint32_t(mf), uint32_t(I32_MIN), imax);
      if (lane == 0) {
        L.red[0][wave] = r0;
        L.red[1][wave] = r1;
        L.red[2][wave] = r2;
      }
    }
    for (int i = tid; i < SBINS; i += RNT) L.hist[i] = 0u;
    if (tid == 0) L.sh_ncand = 0u;
    __syncthreads();
    mn = int32_t(row0_reduce(lane < RWAVES ? L.red[0][lane] : uint32_t(I32_MAX), uint32_t(I32_MAX), imin));
    mx = int32_t(row0_reduce(lane < RWAVES ? L.red[1][lane] : uint32_t(I32_MIN), uint32_t(I32_MIN), imax));
    mf = int32_t(row0_reduce(lane < RWAVES ? L.red[2][lane] : uint32_t(I32_MIN), uint32_t(I32_MIN), imax));
    if (mn < KEY_NINF || mx > KEY_PINF) {
      // some score is NaN: every NaN key becomes KEY_NAN and the extremes are taken again
      // (KEY_NAN + FIN_SHIFT stays clear of INT_MIN)
      mn = I32_MAX;
      mf = I32_MIN;
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        int32_t s = int32_t(key[j]);
        s = (s < KEY_NINF || s > KEY_PINF) ? KEY_NAN : s;
        key[j] = uint32_t(s);
        const bool v = valid(j);
        mn = v ? min(mn, s) : mn;
        mf = v ? max(mf, int32_t(uint32_t(s) + FIN_SHIFT)) : mf;
      }
      const uint32_t r0 = wave_reduce(uint32_t(mn), uint32_t(I32_MAX), imin);
      const uint32_t r2 = wave_reduce(uint32_t(mf), uint32_t(I32_MIN), imax);
      if (lane == 0) {
        L.red[3][wave] = r0;
        L.red[4][wave] = r2;
      }
      __syncthreads();
      mn = int32_t(row0_reduce(lane < RWAVES ? L.red[3][lane] : uint32_t(I32_MAX), uint32_t(I32_MAX), imin));
      mf = int32_t(row0_reduce(lane < RWAVES ? L.red[4][lane] : uint32_t(I32_MIN), uint32_t(I32_MIN), imax));
    }
    // From here on the registers hold rel = min(key - kmin, rcap): the order is unchanged and
    // +inf keys (if any) equal rcap.  With no key below +inf, every rel is 0.  Padding
    // (indices past the end) becomes rel 0, the smallest key: it is last in index order, and
    // since k < n the kept ties (lowest index first) never reach it, so it changes no
    // selection; counts below may include it.
    const uint32_t kmin = uint32_t(mn);
    const uint32_t rcap = mf != I32_MIN ? uint32_t(mf) - FIN_SHIFT - kmin + 1u : 0u;
    if (whole) {
#pragma unroll
      for (int j = 0; j < RPT; ++j) key[j] = min(key[j] - kmin, rcap);
    } else {
#pragma unroll
      for (int j = 0; j < RPT; ++j) key[j] = valid(j) ? min(key[j] - kmin, rcap) : 0u;
    }

    // T: the k-th largest rel; keep `rem` of the keys equal to T, of which there are `cnt`
    // (a count that may include padding)
    uint32_t rem = uint32_t(k), cnt;
    uint32_t prefix = 0u;   // rel >> hi of the keys still in the running
    const int B = rcap ? 32 - __clz(rcap) : 0;   // rel < 2^B
    if (B == 0) {
      cnt = uint32_t(n);   // every key is 0
    } else {
      int hi = B > SD ? B - SD : 0;
      // Chunks wholly past the end hold only padding (rel 0): one thread counts them into
      // bin 0 at once.  Key by key, every lane of such a load's keys would hit that one bin.
#pragma unroll
      for (int c = 0; c < RCH; ++c) {
        if (c * RCHUNK < n) {
#pragma unroll
          for (int u = 0; u < RCW; ++u) atomicAdd(&L.hist[key[RCW * c + u] >> hi], 1u);
        }
      }
      if (tid == 0 && n < RMAX) atomicAdd(&L.hist[0], uint32_t(RCHUNK * (RCH - (n + RCHUNK - 1) / RCHUNK)));
      __syncthreads();
      if (wave == 0) {
        const Pick p = pick_bucket<SBINS / 64>(L.hist, rem, lane);
        if (lane == 0) {
          L.sh_digit = p.digit;
          L.sh_rem = p.rem;
          L.sh_cnt = p.cnt;
        }
      }
      __syncthreads();
      prefix = L.sh_digit;
      rem = L.sh_rem;
      cnt = L.sh_cnt;
      if (hi > 0 && cnt <= uint32_t(CMAX)) {
        // The `cnt` keys of the chosen bucket (rel - cbase < 2^Lb) go to LDS as their low Lb
        // bits.
        const int Lb = hi;
        const uint32_t cbase = prefix << Lb, width = 1u << Lb;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
          // a key enters the list where it finds it (the finish needs no order); the
          // increments of one instruction are combined by a single lane
          const uint32_t d = key[j] - cbase;
          if (d < width) {
            const uint32_t pos = atomicAdd(&L.sh_ncand, 1u);
            if (pos < uint32_t(CMAX)) L.cand[pos] = d;
          }
        }
        __syncthreads();
        if (wave == 0) {
          // radix passes of WD bits over the list, by this wave alone: its LDS operations
          // execute in program order, so the clears, the atomics and the reads of whist
          // need no barrier (the waits and fences keep the compiler from moving them)
          const int nc = int(min(cnt, uint32_t(CMAX)));
          uint32_t p2 = 0u, r2 = rem, c2 = cnt;
          int h2 = Lb;
          while (h2 > 0) {
            const int l2 = h2 > WD ? h2 - WD : 0;
            const uint32_t m2 = (1u << (h2 - l2)) - 1u;
#pragma unroll
            for (int q = 0; q < WBINS / 64; ++q) L.whist[WBINS / 64 * lane + q] = 0u;
            asm volatile("" ::: "memory");
            // eight reads in flight before their atomics: the list is walked at LDS
            // throughput rather than one read latency per element
            for (int i0 = 0; i0 < nc; i0 += 8 * 64) {
              uint32_t vv[8];
#pragma unroll
              for (int u = 0; u < 8; ++u) vv[u] = L.cand[min(i0 + u * 64 + lane, CMAX - 1)];
#pragma unroll
              for (int u = 0; u < 8; ++u)
                if (i0 + u * 64 + lane < nc && (vv[u] >> h2) == p2)
                  atomicAdd(&L.whist[(vv[u] >> l2) & m2], 1u);
            }
            __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
            asm volatile("" ::: "memory");
            const Pick pk = pick_bucket<WBINS / 64>(L.whist, r2, lane);
            __builtin_amdgcn_s_waitcnt(0xc07f);
            asm volatile("" ::: "memory");
            p2 = (p2 << (h2 - l2)) | pk.digit;
            r2 = pk.rem;
            c2 = pk.cnt;
            h2 = l2;
          }
          if (lane == 0) {
            L.sh_digit = p2;
            L.sh_rem = r2;
            L.sh_cnt = c2;
          }
        }
        __syncthreads();
        prefix = (prefix << Lb) | L.sh_digit;
        rem = L.sh_rem;
        cnt = L.sh_cnt;
        hi = 0;
      }
      while (hi > 0) {
        // another block-wide digit over the keys whose bits above hi equal prefix: clear the
        // histogram (the pick above read it before the barrier that ended it)
        for (int i = tid; i < SBINS; i += RNT) L.hist[i] = 0u;
        __syncthreads();
        const int lo = hi > SD ? hi - SD : 0;
        const uint32_t dmask = (1u << (hi - lo)) - 1u;
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
          const uint32_t rel = key[j];
          if ((rel >> hi) == prefix) atomicAdd(&L.hist[(rel >> lo) & dmask], 1u);
          __builtin_amdgcn_sched_barrier(0);   // one key at a time: no 32 live masks
        }
        __syncthreads();
        if (wave == 0) {
          const Pick p = pick_bucket<SBINS / 64>(L.hist, rem, lane);
          if (lane == 0) {
            L.sh_digit = p.digit;
            L.sh_rem = p.rem;
            L.sh_cnt = p.cnt;
          }
        }
        __syncthreads();
        prefix = (prefix << (hi - lo)) | L.sh_digit;
        rem = L.sh_rem;
        cnt = L.sh_cnt;
        hi = lo;
      }
    }
    const uint32_t T = prefix;
    // every tie is kept when their count equals the number still to keep (a count that
    // includes padding cannot: real ties alone already reach rem); keys >= T1 are kept
    // outright
    const bool all_ties = cnt == rem;
    const uint32_t T1 = all_ties ? T : T + 1u;

    uint32_t take = 0u, own[RCH / 2];
    uint32_t base[RCH];
    if (all_ties) {
      // kept: the keys >= T1, counted per chunk (no mask: the stores compare again)
      uint32_t cc[RCH];
#pragma unroll
      for (int c = 0; c < RCH; ++c) {
        cc[c] = 0u;
#pragma unroll
        for (int u = 0; u < RCW; ++u) cc[c] += uint32_t(key[RCW * c + u] >= T1);
      }
#pragma unroll
      for (int q = 0; q < RCH / 2; ++q) own[q] = cc[2 * q] | (cc[2 * q + 1] << 16);
    } else {
      // ties ranked in index order; the first rem are kept
      uint32_t eq = 0u;
#pragma unroll
      for (int j = RPT - 1; j >= 0; --j) {
        take = (take << 1) | uint32_t(key[j] >= T1);
        eq = (eq << 1) | uint32_t(key[j] == T);
      }
      chunk_counts(eq, own);
      chunk_offsets(own, base, L.wtot[0], lane, wave);
#pragma unroll
      for (int j = 0; j < RPT; ++j) {
        const uint32_t below = uint32_t(__popc(eq & (((1u << (j & 3)) - 1u) << (j & ~3))));
        take |= uint32_t(((eq >> j) & 1u) && base[j >> 2] + below < rem) << j;
      }
      chunk_counts(take, own);
    }
    chunk_offsets(own, base, L.wtot[1], lane, wave);
    int t4s = 4 * tid;
    asm volatile("" : "+v"(t4s));
    // kept keys of chunk c at ranks base[c], base[c] + 1, ...; the descriptor's bound (the
    // budget) drops any store past it
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(out, 0, 4 * k, 0x00020000);
    auto emit = [&](auto kept) {
#pragma unroll
      for (int c = 0; c < RCH; ++c) {
        uint32_t r = 4u * base[c];
#pragma unroll
        for (int u = 0; u < RCW; ++u) {
          if (kept(RCW * c + u)) {
            __builtin_amdgcn_raw_buffer_store_b32(uint32_t(c * RCHUNK + t4s + u), rs, int(r), 0, 0);
            r += 4u;
          }
        }
      }
    };
    if (all_ties)
      emit([&](int j) { return key[j] >= T1; });
    else
      emit([&](int j) { return ((take >> j) & 1u) != 0u; });
  }
}

}  // namespace

bool select_regular(const SelSeg* segs_h, int n_segs) {
  if (n_segs < 2) return n_segs == 1;
  const int64_t stride = segs_h[1].start - segs_h[0].start;
  for (int i = 1; i < n_segs; ++i)
    if (segs_h[i].len != segs_h[0].len || segs_h[i].k != segs_h[0].k ||
        segs_h[i].start - segs_h[i - 1].start != stride || segs_h[i].out != int64_t(i) * segs_h[0].k)
      return false;
  return segs_h[0].out == 0;
}

hipError_t launch_select(const float* scores, const SelSeg* segs_h, const SelSeg* segs_d,
                         int n_segs, int max_len, int32_t* keep, hipStream_t s) {
  if (n_segs == 0) return hipSuccess;
  SelInline inl{};
  if (n_segs <= SEL_INLINE) {
    for (int i = 0; i < n_segs; ++i) inl.s[i] = segs_h[i];
    inl.n = n_segs;
  } else if (select_regular(segs_h, n_segs)) {
    // equal segments at a fixed stride (one per KV head over the same scores, a batch of
    // equal-length sequences): the kernels compute each descriptor, nothing is uploaded
    inl.regular = 1;
    inl.start0 = segs_h[0].start;
    inl.stride = segs_h[1].start - segs_h[0].start;
    inl.len = segs_h[0].len;
    inl.k = segs_h[0].k;
  }
  // The register path pays a fixed cost per segment (its passes and scans are a chain of
  // block-wide barriers) that the re-reading kernel does not; it wins once a segment is
  // long enough for the repeated reads to dominate.
  if (max_len > 8192 && max_len <= RMAX) {
    // one workgroup per CU of the current device, each walking segments
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(select_keep_regs, dim3(std::min(n_segs, std::max(cus, 1))), dim3(RNT), 0, s, scores,
                       segs_d, inl, n_segs, keep);
  } else {
    hipLaunchKernelGGL(select_keep_kernel, dim3(n_segs), dim3(SNT), 0, s, scores, segs_d, inl, keep);
  }
  return hipGetLastError();
}

}  // namespace cc
