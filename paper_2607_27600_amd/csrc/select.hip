// Keep selection of the memory-refresh cycle (Sec. 3.2): per segment, the k entries that
// come first under (score descending, ties to the lower index), emitted in ascending
// index order so the compacted cache keeps the original time order.
//
// One workgroup per segment.  Scores map to order-preserving 32-bit keys (-0 == +0, NaN
// below -inf).  Four 8-bit radix passes over the keys (LDS histogram, wave-parallel
// bucket search) find the k-th largest key T and how many entries equal to T are kept;
// a final pass in index order emits every key > T and the lowest-index ties with
// block-wide ballot/prefix counts.  Integer work only: the result is exact.
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
  __shared__ uint32_t sh_digit, sh_rem;
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

  int ties_before = 0, emitted = 0;
  for (int base = 0; base < n; base += SNT) {
    const int i = base + tid;
    const uint32_t key = i < n ? order_key(s[i]) : 0u;
    const bool eq = i < n && key == T;
    const bool gt = i < n && key > T;
    int eq_total;
    const int tie_rank = ties_before + block_scan(eq, wsum, eq_total);
    const bool take = gt || (eq && uint32_t(tie_rank) < rem);
    int take_total;
    const int pos = emitted + block_scan(take, wsum, take_total);
    if (take) out[pos] = i;
    ties_before += eq_total;
    emitted += take_total;
  }
}

}  // namespace

hipError_t launch_select(const float* scores, const SelSeg* segs_d, int n_segs, int max_len,
                         int32_t* keep, hipStream_t s) {
  (void)max_len;
  if (n_segs == 0) return hipSuccess;
  hipLaunchKernelGGL(select_keep_kernel, dim3(n_segs), dim3(SNT), 0, s, scores, segs_d, keep);
  return hipGetLastError();
}

}  // namespace cc
