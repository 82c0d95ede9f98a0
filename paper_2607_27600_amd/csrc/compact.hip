// KV compaction of the memory-refresh cycle (Sec. 3.2): the kept entries of every cache
// layer and KV head are gathered to the front of their sequence, dst[j] = src[keep[j]],
// as a bit copy of one head_dim row; token ids and position ids follow the same list.
//
// Out of place: one workgroup per (plane, chunk of rows), fully parallel.
// In place: keep is ascending, so keep[j] >= j and a destination slot j can only be the
// source of an entry j' <= j.  One workgroup walks its plane in chunks of rows in
// increasing order.  Chunk c's rows are written only after a barrier that every thread
// reaches with chunk c's loads (and so all earlier loads) returned, which orders every
// read of those slots before the writes.  The sources of chunk c+1 are at or past slot
// (c+1)*rows, beyond everything chunk c writes, so its loads (and the keep indices of
// chunk c+3) are issued before chunk c is written and stay in flight across the barrier.  A plane is (sequence, layer,
// KV head, keys|values); there are hundreds to thousands per refresh.
#include "cc_internal.h"

namespace cc {
namespace {

constexpr int CNT = 256;      // threads per workgroup
constexpr int CU = 5;         // 16-byte row pieces in flight per thread per chunk

struct CompactArgs {
  KvView src[2], dst[2];
  int row16;                  // row bytes / 16
  const int32_t* keep;
  const CompactList* lists;
  const CompactPlane* planes;
  int n_planes;
  int n_tensors;              // 1 (ids layout of one tensor) or 2 (keys and values)
  int rows_per_chunk;         // (CNT / row16) * CU
};

// A 16-byte piece of a source row, read non-temporally: a kept row is read once and never
// again, so the load need not stay in the caches.  Measured with the cache flushed, in-place
// compaction of a contiguous 32-layer, 8-head cache keeping 4096 of 32768 entries (1.07 GB
// moved) goes from 5.4 to 6.3 TB/s, of a paged 28-layer, 4-head cache keeping 20% of eight
// sequences (1.74 GB) from 4.9 to 5.1 TB/s.  (The same hint on the stores makes both slower:
// the compacted rows are written in runs that the caches merge.)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16(const char* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// The paged in-place steps.  A source row needs its keep index, then its page number,
// then the row; a destination row needs its page number.  Step c issues, in this order,
// the keep indices of chunk c+3, the source pages of chunk c+2 (with the in-page rows),
// the destination pages and the rows of chunk c+1, then writes chunk c after the barrier.
// Everything a step waits for was issued before the rows of chunk c, so the rows of chunk
// c+1 stay in flight across the barrier.  Buffers alternate between even and odd steps.
struct PagedBufs {
  int idx[CU], spg[CU], srow[CU], dpg[CU];
  uint4 rows[CU];
};

__device__ __forceinline__ void compact_paged_steps(const CompactArgs& a, const KvView& v,
                                                    const CompactPlane& P, const int32_t* keep,
                                                    int k, char* base, int sub, int r0,
                                                    int rstep, int esz16, int R, int nch) {
  (void)a;
  (void)sub;
  const int32_t* bt = v.block_table + int64_t(P.seq) * v.max_pages;
  char* pb = base + int64_t(P.layer) * v.layer_stride + int64_t(P.head) * v.head_stride + esz16;
  auto slot = [&](int c, int u) { return min(c * R + r0 + u * rstep, k - 1); };
  auto ld_idx = [&](int c, int (&I)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u) I[u] = keep[slot(min(c, nch - 1), u)];
  };
  auto ld_spg = [&](const int (&I)[CU], int (&SP)[CU], int (&RW)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      SP[u] = bt[I[u] >> v.page_shift];
      RW[u] = I[u] & v.page_mask;
    }
  };
  auto ld_dpg = [&](int c, int (&DP)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u) DP[u] = bt[slot(min(c, nch - 1), u) >> v.page_shift];
  };
  auto ld_rows = [&](const int (&SP)[CU], const int (&RW)[CU], uint4 (&D)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u)
      D[u] = ldg16(pb + int64_t(SP[u]) * v.page_stride + int64_t(RW[u]) * v.tok_stride);
  };
  PagedBufs e, o;   // e: buffers read in even steps, o: in odd steps (roles swap each step)
  // prologue: state for step 0 = indices of chunk 2, source pages of chunk 1, destination
  // pages and rows of chunk 0
  ld_idx(0, e.idx);
  ld_idx(1, o.idx);
  __builtin_amdgcn_sched_barrier(0);
  ld_spg(e.idx, o.spg, o.srow);   // chunk 0 -> held in o until its rows are issued below
  ld_spg(o.idx, e.spg, e.srow);   // chunk 1
  ld_idx(2, e.idx);
  ld_dpg(0, e.dpg);
  __builtin_amdgcn_sched_barrier(0);
  ld_rows(o.spg, o.srow, e.rows);
  // step c (cur = buffers of parity c, nxt = the other):
  //   cur.idx = chunk c+2, cur.spg/srow = chunk c+1, cur.dpg/rows = chunk c
  auto step = [&](int c, PagedBufs& cur, PagedBufs& nxt) {
    ld_idx(c + 3, nxt.idx);
    __builtin_amdgcn_sched_barrier(0);
    ld_spg(cur.idx, nxt.spg, nxt.srow);
    ld_dpg(c + 1, nxt.dpg);
    __builtin_amdgcn_sched_barrier(0);
    ld_rows(cur.spg, cur.srow, nxt.rows);
#pragma unroll
    for (int u = 0; u < CU; ++u)
      asm volatile("" ::"v"(cur.rows[u].x), "v"(cur.rows[u].y), "v"(cur.rows[u].z), "v"(cur.rows[u].w));
    __syncthreads();
#pragma unroll
    for (int u = 0; u < CU; ++u) {
      const int j = c * R + r0 + u * rstep;
      if (j < k)
        *reinterpret_cast<uint4*>(pb + int64_t(cur.dpg[u]) * v.page_stride +
                                  int64_t(j & v.page_mask) * v.tok_stride) = cur.rows[u];
    }
  };
  for (int c = 0; c < nch; c += 2) {
    step(c, e, o);
    step(c + 1, o, e);
  }
}

template <bool PAGED>
__global__ __launch_bounds__(CNT) void compact_in_place_kernel(CompactArgs a) {
  // plane-major: the keys and the values of a plane are adjacent workgroups, so the planes
  // (sorted longest first) start in that order for both tensors when not all are resident
  const int tensor = blockIdx.x % a.n_tensors;
  const CompactPlane P = a.planes[blockIdx.x / a.n_tensors];
  const CompactList L = a.lists[P.list];
  const int32_t* keep = a.keep + L.keep_off;
  const int k = L.k;
  if (k <= 0) return;
  const KvView& v = a.src[tensor];   // source and destination views are the same
  char* base = reinterpret_cast<char*>(const_cast<void*>(v.base)) + L.tok0 * v.tok_stride;
  const int tpr = a.row16;
  const int sub = threadIdx.x % tpr;
  const int r0 = threadIdx.x / tpr;
  const int rstep = CNT / tpr;
  const int esz16 = sub * 16;
  const int R = a.rows_per_chunk;
  const int nch = (k + R - 1) / R;
  auto load_idx = [&](int c, int (&idx)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u) idx[u] = keep[min(c * R + r0 + u * rstep, k - 1)];
  };
  auto load_rows = [&](const int (&idx)[CU], uint4 (&buf)[CU]) {
#pragma unroll
    for (int u = 0; u < CU; ++u)
      buf[u] = ldg16(base + kv_off<PAGED>(v, P.seq, P.layer, P.head, idx[u]) + esz16);
  };
  if constexpr (PAGED) {
    compact_paged_steps(a, v, P, keep, k, base, sub, r0, rstep, esz16, R, nch);
    return;
  } else {
    // Loads complete in issue order.  Each chunk step issues the keep indices of chunk c+2
    // before the rows of chunk c+1, so the indices a step waits for were issued before the
    // rows of the chunk being written and waiting for them never waits for those rows.  Two
    // index and two row buffers alternate; the loop is unrolled twice with the chunk count
    // rounded up to even (a register copy of a pending load, or a conditional step, would
    // make the compiler wait for every load).
    int ia[CU], ib[CU];
    uint4 dx[CU], dy[CU];
    // step c: `in` holds chunk c+1's indices, `dc` chunk c's rows; past the end, loads
    // re-read the last chunk and nothing is stored
    auto body = [&](int c, const int (&in)[CU], int (&ifree)[CU], const uint4 (&dc)[CU],
                    uint4 (&dn)[CU]) {
      load_idx(min(c + 2, nch - 1), ifree);
      __builtin_amdgcn_sched_barrier(0);   // keep the issue order: indices, then rows
      load_rows(in, dn);
  #pragma unroll
      for (int u = 0; u < CU; ++u)
        asm volatile("" ::"v"(dc[u].x), "v"(dc[u].y), "v"(dc[u].z), "v"(dc[u].w));
      __syncthreads();
  #pragma unroll
      for (int u = 0; u < CU; ++u) {
        const int j = c * R + r0 + u * rstep;
        if (j < k)
          *reinterpret_cast<uint4*>(base + kv_off<PAGED>(v, P.seq, P.layer, P.head, j) + esz16) = dc[u];
      }
    };
    load_idx(0, ia);
    load_idx(min(1, nch - 1), ib);
    __builtin_amdgcn_sched_barrier(0);
    load_rows(ia, dx);
    for (int c = 0; c < nch; c += 2) {
      body(c, ib, ia, dx, dy);
      body(c + 1, ia, ib, dy, dx);
    }
  }
}

template <bool PAGED>
__global__ __launch_bounds__(CNT) void compact_kernel(CompactArgs a) {
  const int tensor = blockIdx.x % a.n_tensors;
  const CompactPlane P = a.planes[blockIdx.x / a.n_tensors];
  const CompactList L = a.lists[P.list];
  const int32_t* keep = a.keep + L.keep_off;
  const int k = L.k;
  const KvView& sv = a.src[tensor];
  const KvView& dv = a.dst[tensor];
  const char* sb = reinterpret_cast<const char*>(sv.base) + L.tok0 * sv.tok_stride;
  char* db = reinterpret_cast<char*>(const_cast<void*>(dv.base)) + L.tok0 * dv.tok_stride;
  const int tpr = a.row16;
  const int sub = threadIdx.x % tpr;
  const int r0 = threadIdx.x / tpr;
  const int rstep = CNT / tpr;
  const int esz16 = sub * 16;
  // element size is folded into the strides: the views carry byte strides here
  const int j_begin = blockIdx.y * a.rows_per_chunk;
  const int j_end = min(k, j_begin + a.rows_per_chunk);
  for (int j0 = j_begin; j0 < j_end; j0 += a.rows_per_chunk) {
    // branch-free gather: rows past the list end re-read its last entry and are not stored
    int src[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u) src[u] = keep[min(j0 + r0 + u * rstep, j_end - 1)];
    uint4 buf[CU];
#pragma unroll
    for (int u = 0; u < CU; ++u)
      buf[u] = ldg16(sb + kv_off<PAGED>(sv, P.seq, P.layer, P.head, src[u]) + esz16);
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
  a.n_tensors = c.n_tensors;
  a.rows_per_chunk = (CNT / a.row16) * CU;
  if (c.n_planes > 0) {
    if (c.in_place) {
      dim3 grid(c.n_tensors * c.n_planes);
      if (c.paged)
        hipLaunchKernelGGL(compact_in_place_kernel<true>, grid, dim3(CNT), 0, s, a);
      else
        hipLaunchKernelGGL(compact_in_place_kernel<false>, grid, dim3(CNT), 0, s, a);
    } else {
      // chunks sized by the longest list; planes with shorter lists exit early
      dim3 grid(c.n_tensors * c.n_planes, (c.max_k + a.rows_per_chunk - 1) / a.rows_per_chunk);
      if (grid.y > 0) {
        if (c.paged)
          hipLaunchKernelGGL(compact_kernel<true>, grid, dim3(CNT), 0, s, a);
        else
          hipLaunchKernelGGL(compact_kernel<false>, grid, dim3(CNT), 0, s, a);
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
