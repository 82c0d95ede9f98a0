// KV compaction of the memory-refresh cycle (Sec. 3.2): the kept entries of every cache
// layer and KV head are gathered to the front of their sequence, dst[j] = src[keep[j]],
// as a bit copy of one head_dim row; token ids and position ids follow the same list.
//
// Out of place: one workgroup per (plane, chunk of rows), fully parallel.
// In place: keep is ascending, so keep[j] >= j and a destination slot j can only be the
// source of an entry j' <= j.  One workgroup walks its plane in chunks of rows in
// increasing order: it loads the whole chunk into registers, waits at a barrier until
// every thread's loads have returned, then writes the chunk.  The next chunk's sources
// are all at or past its own first slot, beyond every slot written so far, so a single
// barrier per chunk orders all reads before the writes that could clobber them.  A plane
// is (sequence, layer, KV head, keys|values); there are thousands per refresh.
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int CNT = 256;      // threads per workgroup
constexpr int CU = 8;         // 16-byte rows pieces in flight per thread per chunk

struct CompactArgs {
  KvView src[2], dst[2];
  int row16;                  // row bytes / 16
  const int32_t* keep;
  const CompactList* lists;
  const CompactPlane* planes;
  int n_planes;
  int rows_per_chunk;         // (CNT / row16) * CU
};

__device__ __forceinline__ uint4 ldg16(const char* p) { return *reinterpret_cast<const uint4*>(p); }

template <bool PAGED, bool IN_PLACE>
__global__ __launch_bounds__(CNT) void compact_kernel(CompactArgs a) {
  const int tensor = blockIdx.x / a.n_planes;
  const CompactPlane P = a.planes[blockIdx.x % a.n_planes];
  const CompactList L = a.lists[P.list];
  const int32_t* keep = a.keep + L.keep_off;
  const int k = L.k;
  const KvView& sv = a.src[tensor];
  const KvView& dv = a.dst[tensor];
  const char* sb = reinterpret_cast<const char*>(sv.base);
  char* db = reinterpret_cast<char*>(const_cast<void*>(dv.base));
  const int tpr = a.row16;
  const int sub = threadIdx.x % tpr;
  const int r0 = threadIdx.x / tpr;
  const int rstep = CNT / tpr;
  const int esz16 = sub * 16;
  // element size is folded into the strides: the views carry byte strides here
  int j_begin = IN_PLACE ? 0 : blockIdx.y * a.rows_per_chunk;
  int j_end = IN_PLACE ? k : min(k, j_begin + a.rows_per_chunk);
  for (int j0 = j_begin; j0 < j_end; j0 += a.rows_per_chunk) {
    // branch-free gather: rows past the list end re-read its last entry and are not stored
    int src[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) src[u] = keep[min(j0 + r0 + u * rstep, j_end - 1)];
    uint4 buf[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u)
      buf[u] = ldg16(sb + kv_off<PAGED>(sv, P.seq, P.layer, P.head, src[u]) + esz16);
    if (IN_PLACE) {
      __builtin_amdgcn_s_waitcnt(0);   // this thread's loads have returned
      __syncthreads();                 // ... and so have everyone's
    }
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const int j = j0 + r0 + u * rstep;
      if (j < j_end)
        *reinterpret_cast<uint4*>(db + kv_off<PAGED>(dv, P.seq, P.layer, P.head, j) + esz16) =
            buf[u];
    }
  }
}

// ids[cu_b + j] = ids[cu_b + keep[j]] in place for one sequence's first list.
__global__ __launch_bounds__(CNT) void compact_ids_kernel(int32_t* ids0, int32_t* ids1,
                                                          const int32_t* cu,
                                                          const int32_t* keep,
                                                          const CompactList* lists,
                                                          const int32_t* seq_list) {
  const int b = blockIdx.x;
  const CompactList L = lists[seq_list[b]];
  const int32_t* kp = keep + L.keep_off;
  const int base = cu[b];
  for (int j0 = 0; j0 < L.k; j0 += CNT) {
    const int j = j0 + threadIdx.x;
    int32_t a0 = 0, a1 = 0;
    if (j < L.k) {
      const int src = base + kp[j];
      if (ids0) a0 = ids0[src];
      if (ids1) a1 = ids1[src];
    }
    __builtin_amdgcn_s_waitcnt(0);   // loads returned before anyone overwrites a source
    __syncthreads();
    if (j < L.k) {
      if (ids0) ids0[base + j] = a0;
      if (ids1) ids1[base + j] = a1;
    }
  }
}

}  // namespace

hipError_t launch_compact(const CompactLaunch& c, hipStream_t s) {
  CompactArgs a;
  for (int t = 0; t < 2; ++t) {
    a.src[t] = c.src[t];
    a.dst[t] = c.dst[t];
  }
  a.row16 = c.row_bytes / 16;
  a.keep = c.keep;
  a.lists = c.lists_d;
  a.planes = c.planes_d;
  a.n_planes = c.n_planes;
  a.rows_per_chunk = (CNT / a.row16) * CU;
  if (c.n_planes > 0) {
    if (c.in_place) {
      dim3 grid(2 * c.n_planes);
      if (c.paged)
        hipLaunchKernelGGL((compact_kernel<true, true>), grid, dim3(CNT), 0, s, a);
      else
        hipLaunchKernelGGL((compact_kernel<false, true>), grid, dim3(CNT), 0, s, a);
    } else {
      // chunks sized by the longest list; planes with shorter lists exit early
      dim3 grid(2 * c.n_planes, (c.max_k + a.rows_per_chunk - 1) / a.rows_per_chunk);
      if (grid.y > 0) {
        if (c.paged)
          hipLaunchKernelGGL((compact_kernel<true, false>), grid, dim3(CNT), 0, s, a);
        else
          hipLaunchKernelGGL((compact_kernel<false, false>), grid, dim3(CNT), 0, s, a);
      }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if ((c.ids[0] || c.ids[1]) && c.n_seqs > 0) {
    hipLaunchKernelGGL(compact_ids_kernel, dim3(c.n_seqs), dim3(CNT), 0, s, c.ids[0], c.ids[1],
                       c.cu_d, c.keep, c.lists_d, c.seq_list_d);
    return hipGetLastError();
  }
  return hipSuccess;
}

}  // namespace cc
