// Counter-causal attention (Eq. (2) under the mask of Sec. 3.1): every cached entry i
// attends only to later entries j > i of its own sequence, reusing the stored keys and
// values.  Output o[i][h] = sum_j softmax_j(scale * q[i][h] . k[j][c]) v[j][c], c = h/g.
//
// bf16 path (head_dim 128 or 64): flash-style, one workgroup of 4 waves per (sequence, KV
// head, block of 128 "rows"), where a row is one (position, query head of the GQA group)
// pair, so the g query heads that share a KV head share every K/V tile staged in LDS.
//   S^T = K Q^T and O^T = V^T P^T on 32x32x16 bf16 MFMA.  Computing the transposed
//   products leaves each lane owning one query row (column of the MFMA output), so the
//   online-softmax statistics and rescaling stay in registers of that lane; the P tile
//   feeds the second MFMA straight from registers.
//   Key tiles entirely at or before the block's first row are never visited (they are
//   masked for every row), so the work per block shrinks towards the end of the
//   sequence; only tiles that straddle the diagonal or the sequence end are masked.
//   K and V tiles go from global memory straight into LDS (no register staging), both
//   row-major with XOR-swizzled 16-byte chunks; the V^T operand of the second product is
//   read with LDS transpose reads.  Both are double buffered with one barrier per tile.
// fp32 path: one thread per row, K/V tiles staged in LDS, exact fp32 online softmax.
#include <type_traits>

#include "cc_internal.h"

namespace cc {
namespace {

constexpr int BN = 64;            // keys per tile
constexpr int ROWS_W = 32;        // rows per wave
constexpr int NWAVES = 4;
constexpr int ROWS = ROWS_W * NWAVES;
constexpr float kRescale = 8.f;   // log2 headroom before the softmax reference max moves

// Shape constants of the bf16 kernel for head dim HD (128 or 64).  A K or V tile is
// BN x HD bf16 in LDS, unpadded, rows of 2 HD bytes in 16-byte chunks whose positions are
// XOR-swizzled by bits of the row (key) index so that the fragment reads hit every bank
// once per 16 lanes:
//   HD = 128 (rows of 256 B = all 64 banks): K chunk c of row r at c ^ (r & 15); V chunk c
//     at c ^ ((r & 3) << 2) (the transpose reads take 4 rows at a time);
//   HD = 64 (rows of 128 B = half the banks, so rows r and r + 1 share no bank): K chunk c
//     at c ^ ((r >> 1) & 7); V chunk c at c ^ (((r >> 1) & 1) << 2).
template <int HD>
struct Shape {
  static_assert(HD == 128 || HD == 64, "head dim 128 or 64");
  static constexpr int TILE = BN * HD;      // elements of one K or V tile (16 or 8 KB)
  static constexpr int ROWB = HD * 2;       // bytes per tile row
  static constexpr int CPR = HD / 8;        // 16-byte chunks per row
  static constexpr int RPW = 64 / CPR;      // rows one wave-wide 1 KB load fills
  static constexpr int NI = BN / (NWAVES * RPW);   // load instructions per wave per tile
  static constexpr int NKS = HD / 16;       // k-steps of S^T = K Q^T
  static constexpr int NDB = HD / 32;       // 32-dim blocks of O^T
  static constexpr int NS = 2 * NKS;        // MFMAs of S^T per tile (two 32-key blocks)
  static constexpr int NPV = 4 * NDB;       // MFMAs of O^T per tile (four 16-key steps)
  __device__ static constexpr int kswz(int r) { return HD == 128 ? (r & 15) : ((r >> 1) & 7); }
  __device__ static constexpr int vswz(int r) {
    return HD == 128 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
  }
};

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_void;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));

struct AttnArgs {
  const u16* q;
  u16* o;
  const int32_t* cu;
  const int4* work;   // null for one sequence: item i is (0, i % nkv, i / nkv)
  KvView k, v;
  int layer;
  int hq, g, nkv;
  float c2;        // scale * log2(e)
  int inclusive;
};

__device__ __forceinline__ uint4 ld16(const u16* p) { return *reinterpret_cast<const uint4*>(p); }

// ds_read_b64_tr_b16: in each group of 16 lanes, lane i receives element i%4 of the 8-byte
// chunks addressed by lanes i/4, 4 + i/4, 8 + i/4 and 12 + i/4 of its group.  With lane
// 4e + c of a group addressing row r0 + e, columns c0 + 4c .. +3 of a row-major tile, lane i
// gets column c0 + i of rows r0 .. r0+3: a transposed 4x16 block.
__device__ __forceinline__ v4i16 ds_read_tr(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p));
}

// A wave-uniform pointer held in scalar registers, so that pointer + 32-bit lane offset
// selects the scalar-base form of the load (no per-lane 64-bit address arithmetic).
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(u >> 32));
  return reinterpret_cast<const char*>((uint64_t(hi) << 32) | lo);
}

// One 16-byte-per-lane global -> LDS DMA: lane l's 16 bytes land at LDS byte address
// lds + 16 l.  Issued through inline asm rather than the builtin: with the builtin in the
// loop the compiler waits for all outstanding LDS reads (lgkmcnt(0)) wherever it waits for
// one, which defeats the fragment reads issued ahead of their MFMAs; through asm it counts
// the reads precisely.  The DMAs are ordered by the explicit waitcnt + barrier that ends
// every tile (and the asm's memory clobber keeps the compiler from moving it).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return uint32_t(reinterpret_cast<uintptr_t>((lds_void*)(p)));
}
// scalar base + per-lane 32-bit offset
__device__ __forceinline__ void dma16(const char* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "s"(lds) : "memory", "m0");
}
// per-lane 64-bit address
__device__ __forceinline__ void dma16(const char* vaddr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(vaddr), "s"(lds) : "memory", "m0");
}

// Page numbers of paged-cache slabs (16 keys, which lie in one page because pages hold a
// power of two >= 16 keys), fetched with scalar loads and waited for at once.  They are
// loaded where no LDS read is outstanding (the end of a step, or the prologue), so the wait
// covers only these loads, which hit the scalar cache (16 consecutive table entries per
// line).  Vector loads of the page numbers would be counted with the tile DMAs, which
// complete in order: waiting for a page number would wait for every DMA issued before it.
__device__ __forceinline__ void page_numbers(const int32_t* p0, const int32_t* p1, int& o0, int& o1) {
  asm volatile("s_load_dword %0, %2, 0x0\n\ts_load_dword %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
               : "=&s"(o0), "=&s"(o1) : "s"(p0), "s"(p1) : "memory");
}
__device__ __forceinline__ void page_numbers(const int32_t* p0, const int32_t* p1, const int32_t* p2,
                                             const int32_t* p3, int& o0, int& o1, int& o2, int& o3) {
  asm volatile("s_load_dword %0, %4, 0x0\n\ts_load_dword %1, %5, 0x0\n\t"
               "s_load_dword %2, %6, 0x0\n\ts_load_dword %3, %7, 0x0\n\ts_waitcnt lgkmcnt(0)"
               : "=&s"(o0), "=&s"(o1), "=&s"(o2), "=&s"(o3)
               : "s"(p0), "s"(p1), "s"(p2), "s"(p3) : "memory");
}

template <int HD, bool PAGED>
__global__ __launch_bounds__(256, 2) void attn_cc_bf16(AttnArgs a) {
  using SH = Shape<HD>;
  constexpr int TILE = SH::TILE, ROWB = SH::ROWB, CPR = SH::CPR, RPW = SH::RPW, NI = SH::NI;
  constexpr int NKS = SH::NKS, NDB = SH::NDB, NS = SH::NS, NPV = SH::NPV;
  // Two K and two V buffers as distinct objects: the compiler can then tell the buffer a
  // DMA is filling from the one being read, and waits for the DMA only where asked.
  __shared__ __attribute__((aligned(1024))) u16 kl0[TILE];
  __shared__ __attribute__((aligned(1024))) u16 kl1[TILE];
  __shared__ __attribute__((aligned(1024))) u16 vl0[TILE];
  __shared__ __attribute__((aligned(1024))) u16 vl1[TILE];

  // work item: from the table, or for one sequence from the block index (row blocks in
  // increasing order, heaviest first, KV heads fastest: the table's order)
  const int4 w = a.work ? a.work[blockIdx.x]
                        : make_int4(0, int(blockIdx.x) % a.nkv, int(blockIdx.x) / a.nkv, 0);
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

  // This lane's query row as the B operand of S^T = K Q^T: NKS k-steps of 16 dims,
  // lane half `hi` holds dims ks*16 + hi*8 .. +7.
  bf16x8 qf[NKS];
  {
    const u16* qp = a.q + (int64_t(seq0 + (valid ? pos : 0)) * a.hq + hq) * HD + hi * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
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
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          *reinterpret_cast<uint2*>(op + db * 32 + jj * 8) = make_uint2(0, 0);
    }
    return;
  }
  // tiles [tb, tm0) and [tm1, te) need the mask; [tm0, tm1) see every key of every row
  const int tm0 = min(te, max(tb, (pos_hi_wg + 1 + BN - 1) / BN));
  const int tm1 = (n % BN == 0) ? te : te - 1;

  // ---- tile DMA (global -> LDS, no registers).  Wave w, instruction i fills the RPW tile
  // rows starting at R = 4 RPW i + RPW w (1 KB): lane l writes row R + l / CPR at 16-byte
  // position l % CPR, and loads the row's chunk (l % CPR) ^ swz(row) there (the swizzles of
  // Shape).  The rows of one instruction lie in one 16-key slab (keys 16 s .. 16 s + 15,
  // s = R / 16); drow = R % 16 + l / CPR is the lane's row within the slab.  Rows past the
  // sequence end are clamped to its last key (their weights are 0 and the clamped data is
  // finite).
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int drow = (RPW * NWAVES > 16 ? (wave * RPW) % 16 : wave * RPW) + lane / CPR;
  const int kch = (lane % CPR) ^ SH::kswz(drow);
  const int vch = (lane % CPR) ^ SH::vswz(drow);
  const char* kbase = reinterpret_cast<const char*>(a.k.base);
  const char* vbase = reinterpret_cast<const char*>(a.v.base);
  const int64_t kts = a.k.tok_stride * 2, vts = a.v.tok_stride * 2;   // bytes per key
  uint32_t klane = uint32_t(drow * kts + kch * 16);
  uint32_t vlane = uint32_t(drow * vts + vch * 16);
  // contiguous caches: the (sequence, layer, head) plane; paged: layer + head part
  const char* kplane = kbase + (PAGED ? int64_t(a.layer) * a.k.layer_stride + int64_t(kvh) * a.k.head_stride
                                      : kv_off<false>(a.k, b, a.layer, kvh, 0)) * 2;
  const char* vplane = vbase + (PAGED ? int64_t(a.layer) * a.v.layer_stride + int64_t(kvh) * a.v.head_stride
                                      : kv_off<false>(a.v, b, a.layer, kvh, 0)) * 2;
  const int32_t* btab = PAGED ? a.k.block_table + int64_t(b) * a.k.max_pages : nullptr;
  const int last_page = PAGED ? (n - 1) >> a.k.page_shift : 0;
  // The 16-key slab of load instruction i (wave-uniform): at HD = 128 the four waves' rows
  // of one instruction form slab i; at HD = 64 waves 0-1 fill slab 2i and waves 2-3 slab
  // 2i + 1.
  auto slab_of = [&](int i) {
    return RPW * NWAVES > 16 ? (RPW * NWAVES / 16) * i + (RPW * wave_u) / 16 : i;
  };
  // Page numbers of this wave's slabs of tile t (paged caches; K and V share the block
  // table): scalar loads, waited for at once.  Slabs past the sequence end take its last page.
  auto load_pages = [&](int t, int (&pg)[NI]) {
    if constexpr (PAGED) {
      const int32_t* pp[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) pp[i] = btab + min((t * BN + 16 * slab_of(i)) >> a.k.page_shift, last_page);
      if constexpr (NI == 4)
        page_numbers(pp[0], pp[1], pp[2], pp[3], pg[0], pg[1], pg[2], pg[3]);
      else
        page_numbers(pp[0], pp[1], pg[0], pg[1]);
    }
  };
  // Fill an LDS tile with tile t.  Full tiles of a contiguous cache: from a running tile
  // pointer (tile_ptr = plane + t * BN keys, advanced once per tile), a 64-bit scalar add per
  // 16-key slab and the lane's fixed offset.  Full tiles of a paged cache: a uniform base per
  // slab from its page, pg (loaded beforehand by load_pages).  The last, partial tile:
  // per-lane rows (clamped), per-lane page lookups.
  auto issue = [&](u16* dst, int t, const KvView& kv, const char* plane, const char* tile_ptr,
                   uint32_t lane_off, int ch, int64_t ts, const int (&pg)[NI]) {
    const int key0 = t * BN;
    u16* lds = dst + wave_u * RPW * HD;
    const uint32_t pstride = uint32_t(kv.page_stride * 2);   // bytes per page
    if (key0 + BN <= n) {
      // keep the 32-bit offset opaque here so that it is not widened outside the loop
      asm volatile("" : "+v"(lane_off));
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int si = slab_of(i);
        const char* base;
        if constexpr (PAGED)   // a page spans < 4 GiB: 32 x 32 -> 64-bit page offset
          base = uniform_ptr(plane + (uint64_t(uint32_t(pg[i])) * pstride +
                                      uint32_t((key0 + 16 * si) & kv.page_mask) * uint32_t(ts)));
        else
          base = tile_ptr + int64_t(16 * si) * ts;
        dma16(base, lane_off, lds_addr(lds + i * NWAVES * RPW * HD));
      }
    } else {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int key = min(key0 + 16 * slab_of(i) + drow, n - 1);
        int64_t off;
        if constexpr (PAGED)
          off = int64_t(btab[key >> kv.page_shift]) * kv.page_stride + int64_t(key & kv.page_mask) * kv.tok_stride;
        else
          off = int64_t(key) * kv.tok_stride;
        dma16(plane + off * 2 + ch * 16, lds_addr(lds + i * NWAVES * RPW * HD));
      }
    }
  };

  // ---- fragment reads.  K (A operand of S^T = K Q^T): MFMA j reads row (j&1)*32 + col,
  // chunk 2*(j>>1) + hi.  V^T (A operand of O^T = V^T P^T): MFMA j = (k-step kk, d block db)
  // = (j / NDB, j % NDB) needs d = 32 db + col and keys 16kk + 4hi + {0..3},
  // 16kk + 8 + 4hi + {0..3} (the order of the P operand's k-slots): two transpose reads of
  // 4 keys x 16 dims.  Lane 4y + c of lane group G reads key row 4 (G >> 1) + y at dims
  // 32 db + 16 (G & 1) + 4 c .. +3, i.e. 8-byte half (c & 1) of chunk
  // 4 db + 2 (G & 1) + (c >> 1), at that chunk's swizzled position.
  uint32_t koff[NKS];
#pragma unroll
  for (int jj = 0; jj < NKS; ++jj) koff[jj] = col * ROWB + 16 * ((2 * jj + hi) ^ SH::kswz(col));
  uint32_t voff[NDB];
  {
    const int G = lane >> 4, L = lane & 15, y = L >> 2;
    const int r = 4 * (G >> 1) + y;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      if constexpr (HD == 128)   // vswz(r) = 4 y: the swizzle moves whole 64-byte groups
        voff[db] = r * ROWB + 64 * (db ^ y) + 32 * (G & 1) + 8 * (L & 3);
      else
        voff[db] = r * ROWB + 16 * ((4 * db + 2 * (G & 1) + ((L & 3) >> 1)) ^ SH::vswz(r)) +
                   8 * (L & 1);
    }
  }
  auto kfrag = [&](const u16* Kl, int j) {
    return as_bf16x8(*reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(Kl) +
                                                     koff[j >> 1] + (j & 1) * (32 * ROWB)));
  };
  auto vfrag = [&](const u16* Vl, int j) {
    const char* p = reinterpret_cast<const char*>(Vl) + voff[j % NDB] + (j / NDB) * (16 * ROWB);
    const v4i16 lo = ds_read_tr(p), hi2 = ds_read_tr(p + 8 * ROWB);
    const v8i16 both = __builtin_shufflevector(lo, hi2, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, both);
  };

  // max over both lane halves (they hold the two 32-key blocks of one row)
  auto half_max = [](float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  };
  auto row_max = [&](const f32x16(&s)[2]) {
    float m = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, s[mb][e]);
    return half_max(m);
  };
  auto apply_mask = [&](f32x16(&s)[2], int t) {
    const int key0 = t * BN;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = key0 + mb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
        const bool ok = key < n && (a.inclusive ? key >= pos : key > pos);
        s[mb][e] = ok ? s[mb][e] : -INFINITY;
      }
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};

  // contiguous caches: tile pointers of the next K (t + 2) and V (t + 1) DMAs, in bytes
  const int64_t kstep = int64_t(BN) * kts, vstep = int64_t(BN) * vts;
  const char* kptr = kplane + int64_t(tb + 2) * kstep;
  const char* vptr = vplane + int64_t(tb + 1) * vstep;
  // Paged caches: the page numbers of the tiles the next step loads are fetched at the end
  // of the step before (a tile's K pages are the next step's V pages), so no step waits for
  // a scalar load before its DMAs.  kpg: pages of tile t + 2 (K), vpg: of tile t + 1 (V).
  int kpg[NI], vpg[NI];
  // prologue: K(tb), V(tb), K(tb+1) in LDS; S(tb) and its unmasked row max in registers.
  load_pages(tb, kpg);
  issue(kl0, tb, a.k, kplane, kplane + int64_t(tb) * kstep, klane, kch, kts, kpg);
  issue(vl0, tb, a.v, vplane, vplane + int64_t(tb) * vstep, vlane, vch, vts, kpg);
  load_pages(tb + 1, vpg);
  if (tb + 1 < te) issue(kl1, tb + 1, a.k, kplane, kplane + int64_t(tb + 1) * kstep, klane, kch, kts, vpg);
  if (tb + 2 < te) load_pages(tb + 2, kpg);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  f32x16 sa[2], sb[2];
  sa[0] = f32x16{};
  sa[1] = f32x16{};
#pragma unroll
  for (int j = 0; j < NS; ++j) sa[j & 1] = mfma32(kfrag(kl0, j), qf[j >> 1], sa[j & 1]);
  float mx = row_max(sa);

  // Tile t with parity P = (t - tb) & 1.  S(t) is in sc with its unmasked row max in mx;
  // K(t+1) in kl[1-P], V(t) in vl[P].  The DMAs of K(t+2) -> kl[P] and V(t+1) -> vl[1-P]
  // refill buffers freed by the previous tile.  Issue order: the NS MFMAs of S(t+1) carry
  // the 32 exponentials of tile t; the NPV MFMAs of P V carry the bf16 packing of P, the row
  // sums and the row max of S(t+1).  sched_barrier fences keep the compiler from regrouping.
  auto step = [&](int t, auto par, bool masked) {
    constexpr int P = decltype(par)::value;
    f32x16(&sc)[2] = P ? sb : sa;
    f32x16(&sn)[2] = P ? sa : sb;
    const u16* Kn = P ? kl0 : kl1;
    u16* Kfree = P ? kl1 : kl0;
    const u16* Vc = P ? vl1 : vl0;
    u16* Vfree = P ? vl0 : vl1;
    // tiles past the last are never read: nothing to load
    if (t + 2 < te) issue(Kfree, t + 2, a.k, kplane, kptr, klane, kch, kts, kpg);
    if (t + 1 < te) issue(Vfree, t + 1, a.v, vplane, vptr, vlane, vch, vts, vpg);
    kptr += kstep;
    vptr += vstep;
    bf16x8 kf[4];
    kf[0] = kfrag(Kn, 0);
    kf[1] = kfrag(Kn, 1);
    kf[2] = kfrag(Kn, 2);
    if (masked) {
      apply_mask(sc, t);
      mx = row_max(sc);
    }
    // Lazy rescaling: the reference max only moves when the row max grows by more than
    // 2^8 in probability units (or on the first non-empty tile).  Numerator and
    // denominator always share the reference, so the result is unchanged; p stays <= 256.
    const bool up = mx > m_run + kRescale / a.c2;
    const float corr = up ? fast_exp2((m_run - mx) * a.c2) : 1.f;   // 0 when m_run = -inf
    m_run = up ? mx : m_run;
    const float mc = (m_run == -INFINITY ? 0.f : m_run) * a.c2;
    sn[0] = f32x16{};
    sn[1] = f32x16{};
    __builtin_amdgcn_sched_barrier(0);
    // The section that carries the exponentials issues at raised wave priority, so that on a
    // SIMD shared with a wave in another section its MFMAs and exponentials go first
    // (measured: 4-7% faster at n = 4096, 1.5% at 32768; the same priority over both
    // sections, or over the P V section, gains less or nothing).
    __builtin_amdgcn_s_setprio(1);
    constexpr int EPM = 32 / NS;   // exponentials per MFMA
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      if (j + 3 < NS) kf[(j + 3) & 3] = kfrag(Kn, j + 3);
      sn[j & 1] = mfma32(kf[j & 3], qf[j >> 1], sn[j & 1]);
#pragma unroll
      for (int u = 0; u < EPM; ++u) {
        const int f = EPM * j + u, mb = f >> 4, e = f & 15;
        const float p = fast_exp2(fmaf(sc[mb][e], a.c2, -mc));
        // pin the exponential here, between the MFMAs, instead of next to its later uses
        asm volatile("" ::"v"(p));
        sc[mb][e] = p;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (__any(corr != 1.f)) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) acc[db] *= corr;
    }
    // P^T operand: k-step kk covers keys 16kk .. 16kk+15; lane half hi holds keys
    // {4hi..4hi+3, 8+4hi..8+4hi+3} of that step, i.e. S^T entries 8*(kk%2)..+7 of block kk/2
    bf16x8 pf[4];
    auto pack = [&](int kk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[kk][e] = (__bf16)sc[kk >> 1][(kk & 1) * 8 + e];
    };
    bf16x8 vf[4];
    vf[0] = vfrag(Vc, 0);
    vf[1] = vfrag(Vc, 1);
    vf[2] = vfrag(Vc, 2);
    __builtin_amdgcn_s_setprio(0);
    pack(0);
    float ls0 = 0.f, ls1 = 0.f, m0 = -INFINITY, m1 = -INFINITY;
    constexpr int SPM = 32 / NPV;   // row-sum terms per MFMA
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < NPV; ++j) {
      if (j + 3 < NPV) vf[(j + 3) & 3] = vfrag(Vc, j + 3);
      acc[j % NDB] = mfma32(vf[j & 3], pf[j / NDB], acc[j % NDB]);
      if (j % NDB == NDB - 1 && j < NPV - 1) pack(j / NDB + 1);
#pragma unroll
      for (int u = 0; u < SPM; u += 2) {
        ls0 += sc[(SPM * j + u) >> 4][(SPM * j + u) & 15];
        ls1 += sc[(SPM * j + u + 1) >> 4][(SPM * j + u + 1) & 15];
      }
      asm volatile("" : "+v"(ls0), "+v"(ls1));
      if constexpr (HD == 64) {
        // row max of S(t+1) over slots 2..7: six entries per slot (sn[0] then sn[1])
        if (j >= 2) {
#pragma unroll
          for (int u = 0; u < 6; ++u) {
            const int f = 6 * (j - 2) + u;
            if (f < 16) m0 = fmaxf(m0, sn[0][f]);
            else if (f < 32) m1 = fmaxf(m1, sn[1][f - 16]);
          }
          asm volatile("" : "+v"(m0), "+v"(m1));
        }
      } else if (j >= 2) {
        // row max of S(t+1), whose MFMAs were issued during the exponentials: 32 entries
        // over slots 2..12
        const int f = j - 2;
        if (f < 4) {
          m0 = fmaxf(m0, fmaxf(sn[0][3 * f], fmaxf(sn[0][3 * f + 1], sn[0][3 * f + 2])));
        } else if (f < 5) {
          m0 = fmaxf(m0, fmaxf(sn[0][12], fmaxf(sn[0][13], sn[0][14])));
          m1 = fmaxf(m1, sn[0][15]);
        } else if (f < 10) {
          const int e0 = 3 * (f - 5);
          m1 = fmaxf(m1, fmaxf(sn[1][e0], fmaxf(sn[1][e0 + 1], sn[1][e0 + 2])));
        } else if (f < 11) {
          m1 = fmaxf(m1, sn[1][15]);
        }
        asm volatile("" : "+v"(m0), "+v"(m1));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    l_run = l_run * corr + (ls0 + ls1);
    mx = half_max(fmaxf(m0, m1));
    if constexpr (PAGED) {
      // pages of the next step's tiles; no LDS read is outstanding here, so the loads' wait
      // overlaps the DMA wait below
#pragma unroll
      for (int i = 0; i < NI; ++i) vpg[i] = kpg[i];
      if (t + 3 < te) load_pages(t + 3, kpg);
    }
    __builtin_amdgcn_s_waitcnt(0);   // this wave's DMAs have landed
    __syncthreads();                 // everyone's, and everyone is done with K(t+1), V(t)
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  for (int t = tb; t < te; t += 2) {
    step(t, I0{}, t < tm0 || t >= tm1);
    if (t + 1 < te) step(t + 1, I1{}, t + 1 < tm0 || t + 1 >= tm1);
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  // The output goes out through LDS as whole rows.  The K buffers are free here (the last
  // step waited for every load and ended with a barrier); each wave stages its 32 rows x HD
  // dims (16-byte chunk c of row r at chunk c ^ kswz(r), so the 16-byte row reads hit every
  // bank once, and at HD = 128 the 8-byte writes of the lane halves too), then writes 16
  // bytes per lane along the rows.  The g rows of one position are adjacent in o
  // (head-major), so a wave instruction stores 1 KB of whole rows instead of 64 scattered
  // 8-byte pieces.  LDS operations of one wave complete in order, so the wave needs no
  // barrier of its own.
  char* stg = reinterpret_cast<char*>(wave < 2 ? kl0 : kl1) + (wave & 1) * (ROWS_W * ROWB);
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      bf16x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = (__bf16)(acc[db][jj * 4 + e] * inv);
      const int c = db * 4 + jj;
      *reinterpret_cast<bf16x4*>(stg + col * ROWB + ((c ^ SH::kswz(col)) * 16) + hi * 8) = o;
    }
#pragma unroll
  for (int i = 0; i < ROWS_W * CPR / 64; ++i) {
    const int r = RPW * i + lane / CPR, c = lane % CPR;
    const uint4 v = *reinterpret_cast<const uint4*>(stg + r * ROWB + ((c ^ SH::kswz(r)) * 16));
    const int orow = rb * ROWS + wave * ROWS_W + r;
    if (orow < nrows) {
      const int opos = orow / g, ohq = kvh * g + orow % g;
      *reinterpret_cast<uint4*>(a.o + (int64_t(seq0 + opos) * a.hq + ohq) * HD + c * 8) = v;
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
  const int4* work;   // null for one sequence: item i is (0, i % nkv, i / nkv)
  KvView k, v;
  int layer;
  int hq, g, nkv;
  float scale;
  int inclusive;
};

template <int D, bool PAGED>
__global__ __launch_bounds__(F_ROWS) void attn_cc_f32(AttnArgsF a) {
  __shared__ float Ks[F_BN][D + 1];
  __shared__ float Vs[F_BN][D + 1];
  // work item: from the table, or for one sequence from the block index (row blocks in
  // increasing order, heaviest first, KV heads fastest: the table's order)
  const int4 w = a.work ? a.work[blockIdx.x]
                        : make_int4(0, int(blockIdx.x) % a.nkv, int(blockIdx.x) / a.nkv, 0);
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
  x.nkv = a.n_heads_kv;
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
    if (a.head_dim == 64) {
      if (a.paged)
        hipLaunchKernelGGL((attn_cc_bf16<64, true>), dim3(a.n_work), dim3(256), 0, s, x);
      else
        hipLaunchKernelGGL((attn_cc_bf16<64, false>), dim3(a.n_work), dim3(256), 0, s, x);
    } else {
      if (a.paged)
        hipLaunchKernelGGL((attn_cc_bf16<128, true>), dim3(a.n_work), dim3(256), 0, s, x);
      else
        hipLaunchKernelGGL((attn_cc_bf16<128, false>), dim3(a.n_work), dim3(256), 0, s, x);
    }
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
