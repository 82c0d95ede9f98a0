// Keep selection of the memory-refresh cycle (Sec. 3.2): per segment, the k entries that
// come first under (score descending, ties to the lower index), emitted in ascending
// index order so the compacted cache keeps the original time order.
//
// One workgroup per segment.  Scores map to order-preserving 32-bit keys (-0 == +0, NaN
// below -inf).  8-bit radix passes over the keys (LDS histograms, wave-parallel bucket
// search) find the k-th largest key T and how many entries equal to T are kept; a final
// pass in index order emits every key > T and the lowest-index ties with block-wide
// ballot/prefix counts.  Integer work only: the result is exact.  Launches whose longest
// segment holds 8193..32768 scores keep every segment in registers (one read of the
// scores); the others re-read the scores from memory at every pass.
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int SNT = 1024;           // threads per segment
constexpr int SWAVES = SNT / 64;

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
                                                          int32_t* __restrict__ keep) {
  __shared__ uint32_t hist[256];
  __shared__ int wsum[SWAVES];
  __shared__ uint32_t sh_digit, sh_rem, sh_cnt;
  const SelSeg sg = segs[blockIdx.x];
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
      uint32_t incl = sum;   // inclusive scan over lanes (descending digit order)
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
      }
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
// Segments of up to RMAX scores: the workgroup reads its segment once, coalesced, into
// registers (score j*RNT + t in slot j of thread t) and never touches it again.  The
// radix passes run on rel = key - kmin (kmin, kmax: the segment's extreme keys) over the
// B = bit length of kmax - kmin bits, so the first digit spreads over the scores' actual
// range instead of the few sign and exponent patterns they share.  Histograms are private
// to each wave (fewer colliding LDS atomics) and double buffered (the next pass's buffer
// is cleared while this one is reduced).  The emission ranks ties and kept entries in
// index order from per-(wave, slot) ballot counts, scanned once per kind.
constexpr int RNT = 1024;
constexpr int RWAVES = RNT / 64;
constexpr int RPT = 32;
constexpr int RMAX = RNT * RPT;

// Exclusive scan, in place, of tab[w][j] in (slot j, wave w) order; run by wave 0.
__device__ __forceinline__ void scan_slots(uint32_t (*tab)[RPT], int lane) {
  // lane l takes slots j = l/2 (waves 8*(l&1) .. +7): consecutive lanes follow the order
  const int j = lane >> 1, w0 = (lane & 1) * 8;
  uint32_t v[8], sum = 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v[i] = tab[w0 + i][j];
    sum += v[i];
  }
  uint32_t incl = sum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(incl, off);
    if (lane >= off) incl += t;
  }
  uint32_t run = incl - sum;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    tab[w0 + i][j] = run;
    run += v[i];
  }
}

__global__ __launch_bounds__(RNT, 2) void select_keep_regs(const float* __restrict__ scores,
                                                           const SelSeg* __restrict__ segs,
                                                           int32_t* __restrict__ keep) {
  __shared__ uint32_t hist[2][RWAVES][256];
  __shared__ uint32_t tot[256];
  __shared__ __attribute__((aligned(16))) uint32_t tab[RWAVES][RPT];
  __shared__ uint32_t red[2][RWAVES];
  __shared__ uint32_t sh_digit, sh_rem, sh_cnt;
  const SelSeg sg = segs[blockIdx.x];
  const int n = sg.len, k = sg.k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t* out = keep + sg.out;
  if (k <= 0) return;
  if (k >= n) {
    for (int i = tid; i < n; i += RNT) out[i] = i;
    return;
  }
  // one coalesced read (indices past the end re-read the last score; they never count)
  const float* s = scores + sg.start;
  uint32_t key[RPT];
#pragma unroll
  for (int j = 0; j < RPT; ++j) key[j] = __float_as_uint(s[min(j * RNT + tid, n - 1)]);
#pragma unroll
  for (int j = 0; j < RPT; ++j) key[j] = order_key(__uint_as_float(key[j]));
  const int nvalid = min(RPT, max(0, (n - tid + RNT - 1) / RNT));   // slots j < nvalid hold scores
  auto valid = [&](int j) { return j < nvalid; };

  // extreme keys of the segment; the first histogram buffer is cleared meanwhile
  uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < RPT; ++j)
    if (valid(j)) {
      kmin = min(kmin, key[j]);
      kmax = max(kmax, key[j]);
    }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    kmin = min(kmin, uint32_t(__shfl_xor(kmin, off)));
    kmax = max(kmax, uint32_t(__shfl_xor(kmax, off)));
  }
  if (lane == 0) {
    red[0][wave] = kmin;
    red[1][wave] = kmax;
  }
  for (int i = tid; i < RWAVES * 256; i += RNT) (&hist[0][0][0])[i] = 0u;
  __syncthreads();
  kmin = red[0][0];
  kmax = red[1][0];
#pragma unroll
  for (int w = 1; w < RWAVES; ++w) {
    kmin = min(kmin, red[0][w]);
    kmax = max(kmax, red[1][w]);
  }
  const uint32_t range = kmax - kmin;
  const int B = range ? 32 - __clz(range) : 0;
  // Slots at or past jmax hold no score for any thread and are skipped (a uniform test).
  // The padding of the last, partial slot becomes copies of the smallest key: it is last
  // in index order, and since k < n the kept ties (lowest index first) never reach it, so
  // it changes no selection.
  const int jmax = (n + RNT - 1) / RNT;
#pragma unroll
  for (int j = 0; j < RPT; ++j) key[j] = valid(j) ? key[j] : kmin;

  // radix passes, 8 bits at a time from bit B down; `prefix` holds rel >> hi
  uint32_t prefix = 0u, rem = uint32_t(k);
  int buf = 0;
  for (int hi = B; hi > 0; buf ^= 1) {
    const int lo = hi > 8 ? hi - 8 : 0;
    const uint32_t dmask = (1u << (hi - lo)) - 1u;
    uint32_t(*h)[256] = hist[buf];
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const uint32_t rel = key[j] - kmin;
      const uint32_t top = hi >= 32 ? 0u : rel >> hi;
      if (j < jmax && top == prefix) atomicAdd(&h[wave][(rel >> lo) & dmask], 1u);
    }
    __syncthreads();
    if (tid < 256) {
      uint32_t t = 0u;
#pragma unroll
      for (int w = 0; w < RWAVES; ++w) t += h[w][tid];
      tot[tid] = t;
    }
    for (int i = tid; i < RWAVES * 256; i += RNT) (&hist[buf ^ 1][0][0])[i] = 0u;
    __syncthreads();
    if (tid < 64) {
      // lane l owns digits 255-4l .. 252-4l (descending); find the bucket holding the
      // rem-th largest candidate
      uint32_t c[4], sum = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        c[q] = tot[255 - 4 * lane - q];
        sum += c[q];
      }
      uint32_t incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(incl, off);
        if (lane >= off) incl += t;
      }
      const uint32_t excl = incl - sum;
      if (excl < rem && incl >= rem) {
        uint32_t acc = excl;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (acc + c[q] >= rem) {
            sh_digit = uint32_t(255 - 4 * lane - q);
            sh_rem = rem - acc;
            sh_cnt = c[q];
            break;
          }
          acc += c[q];
        }
      }
    }
    __syncthreads();
    prefix = (prefix << (hi - lo)) | sh_digit;
    rem = sh_rem;
    hi = lo;
  }
  const uint32_t T = kmin + prefix;   // the k-th largest key; keep `rem` of the keys equal to T
  // keys equal to T: the last pass's bucket (all keys when the range is 0).  The count may
  // include padding copies of kmin, so equality with rem proves every tie is kept.
  const bool all_ties = B > 0 && sh_cnt == rem;

  // ranks in index order: element (j, t) comes after every element of slots < j and after
  // (j, t') for t' < t.  A wave's count per slot is a ballot popcount; lane j of each wave
  // records slot j's count and the (slot, wave) table is scanned once; tab[wave][j] is
  // then the number of flagged elements before this wave's part of slot j.
  auto slot_offsets = [&](uint32_t bits) {
    uint32_t mine = 0u;
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
      const uint32_t c = __popcll(__ballot((bits >> j) & 1u));
      mine = lane == j ? c : mine;
    }
    __syncthreads();   // earlier readers of the table are done
    if (lane < RPT) tab[wave][lane] = mine;
    __syncthreads();
    if (wave == 0) scan_slots(tab, lane);
    __syncthreads();
  };
  const uint64_t below = (1ull << lane) - 1ull;
  uint32_t eq_bits = 0u, take_bits = 0u;
#pragma unroll
  for (int j = 0; j < RPT; ++j) {
    eq_bits |= uint32_t(j < jmax && key[j] == T) << j;
    take_bits |= uint32_t(j < jmax && key[j] > T) << j;
  }
  // slots go in groups of four (one wide table read each); the fences keep the compiler
  // from hoisting every group's reads and ballots at once
  if (all_ties) {
    take_bits |= eq_bits;
  } else {
    slot_offsets(eq_bits);
#pragma unroll
    for (int q = 0; q < RPT / 4; ++q) {
      const uint4 o = *reinterpret_cast<const uint4*>(&tab[wave][4 * q]);
      const uint32_t ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int j = 4 * q + e;
        const uint32_t rank = ov[e] + __popcll(__ballot((eq_bits >> j) & 1u) & below);
        take_bits |= uint32_t(((eq_bits >> j) & 1u) && rank < rem) << j;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  slot_offsets(take_bits);
#pragma unroll
  for (int q = 0; q < RPT / 4; ++q) {
    const uint4 o = *reinterpret_cast<const uint4*>(&tab[wave][4 * q]);
    const uint32_t ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int j = 4 * q + e;
      const uint32_t pos = ov[e] + __popcll(__ballot((take_bits >> j) & 1u) & below);
      if (((take_bits >> j) & 1u) && pos < uint32_t(k))   // pos < k always; bounds the store
        out[pos] = j * RNT + tid;
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

}  // namespace

hipError_t launch_select(const float* scores, const SelSeg* segs_d, int n_segs, int max_len,
                         int32_t* keep, hipStream_t s) {
  if (n_segs == 0) return hipSuccess;
  // The register path pays a fixed cost per segment (its passes and scans are a chain of
  // block-wide barriers) that the re-reading kernel does not; it wins once a segment is
  // long enough for the repeated reads to dominate.
  if (max_len > 8192 && max_len <= RMAX)
    hipLaunchKernelGGL(select_keep_regs, dim3(n_segs), dim3(RNT), 0, s, scores, segs_d, keep);
  else
    hipLaunchKernelGGL(select_keep_kernel, dim3(n_segs), dim3(SNT), 0, s, scores, segs_d, keep);
  return hipGetLastError();
}

}  // namespace cc
