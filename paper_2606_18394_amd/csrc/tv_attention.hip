// Tree-verification attention for CDNA4 (gfx950).
//
// Computes, for every draft-tree node v of every sequence and every query
// head, softmax(q_v K^T * scale + M_v) V over the sequence's cached prefix
// and the tree nodes, where the tree-causal mask M_v keeps only v's
// ancestors and v itself (Sec. 2.2, tree-causal mask and masked attention
// equations).  The ancestor relation is rebuilt inside each workgroup as a
// bitmask in LDS from the parent array; no dense mask ever exists (App. E).
//
// Work decomposition.  Rows of one (sequence b, KV head g) pair are the N*G
// (node, head-in-group) pairs, row r = node * G + head.  Keys are cut into
// 32-key tiles: ceil(kv_len/32) cache tiles, then the tree tiles up to the
// last node of the row block (a node never sees a later node because
// parents precede children).  The tiles are cut into S contiguous chunks of
// a fixed size (split-KV).  A workgroup takes one block of 32*WR rows and
// one chunk with WR x WK wave64s: WR row groups of 32 rows, and WK key
// groups that share out the chunk's tiles, each streaming its tiles through
// an LDS ring of NS stages; key groups merge their softmax states in LDS at
// the end.  The host plan (tv_plan.h) picks WR, WK, NS and S per shape so
// that every CU holds 8 waves (two per SIMD).  The prologue requests the
// parents, the queries and every ring stage before it uses any of them;
// with several key groups on a full grid, key group 0 alone loads the
// queries and hands them to the others through LDS.
//
// Per tile.  K and V move HBM -> LDS with global_load_lds_dwordx4 (no
// register staging), rows XOR-swizzled in 16-byte chunks so the transposing
// V reads are free of bank conflicts and the K reads at most two-way (see
// TileLayout).  A wave computes S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16 (keys on the M side, its 32 rows on the N side),
// runs an fp32 base-2 online softmax on the accumulators with a lazily moved
// reference maximum, and accumulates O^T += V^T P^T: P^T comes straight from
// the S^T accumulators (the 32 keys are ordered so the B operand needs no
// data movement) and V^T from ds_read_b64_tr_b16 transposing reads.
//
// Split-KV merge (S > 1).  Every chunk stores its (max, sum, O) partial.
// When one workgroup can merge a row block with at most two batches of
// loads, the chunk that finishes last does it inside this kernel (arrival
// counters in the workspace); otherwise a second kernel merges all row
// blocks.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv_plan.h"

namespace tv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

struct AttnArgs {
  const __bf16* q;
  const __bf16* kc;
  const __bf16* vc;
  const __bf16* kt;
  const __bf16* vt;
  const int32_t* parent;
  const int32_t* kv_len;
  __bf16* out;
  f32x4* ws_o;
  float2* ws_ml;
  unsigned int* arrived;  // per row block: chunks that have stored partials
  int* tree_bad;          // per row block: invalid parent array seen
  int B, N, Hq, Hkv, Lmax, G, M, nRB, S, chunk, nwork;
  int fused;   // split-KV merge inside the main kernel (else a second kernel)
  int spread;  // work order of several sequences (tv_plan.h, work_item)
  float c;  // scale * log2(e): scores live in base-2 exponent units
  const int32_t* block_table;  // paged cache: [B, max_blocks], else NULL
  int block_shift, max_blocks, num_blocks;
  int tail;    // tree-tail layout: node i's K/V are cache row kv_len + i
  int cgroup;  // sequences sharing one cache (sequence b reads cache b / cgroup)
};

// The keys a sequence's row block attends over.  Separate tree K/V: nct
// cache tiles (rows < kvl) then the tree tiles of nodes 0..i_hi.  Tree-tail
// layout: the tree rows follow the context in the cache (kvl is clamped to
// Lmax - N so they fit) and one run of nct = T tiles covers rows
// 0 .. kvl + i_hi.  A NULL kv_len means full caches.
struct Segment {
  int kvl, nct, T;
};
__device__ __forceinline__ Segment segment(const AttnArgs& a, int b, int i_hi) {
  const int cap = a.tail ? a.Lmax - a.N : a.Lmax;
  int kvl = a.kv_len ? a.kv_len[b] : cap;
  kvl = kvl < 0 ? 0 : (kvl > cap ? cap : kvl);
  Segment sg;
  sg.kvl = kvl;
  if (a.tail) {
    sg.nct = (kvl + i_hi + kKeyTile) / kKeyTile;
    sg.T = sg.nct;
  } else {
    sg.nct = (kvl + kKeyTile - 1) / kKeyTile;
    sg.T = sg.nct + i_hi / kKeyTile + 1;
  }
  return sg;
}

// Longest-first order of a ragged batch (spread = 2).  XCD x serves one KV
// head and lane x / Hkv of L = 8 / Hkv lanes of chunks; pair p of the lane
// is sequence p / (S / L) and its (p % (S / L))-th chunk in that lane, as in
// work_item.  Each pair gets the distinct key (tile count << 16 | 0xFFFF - p)
// (longest first, lower pair index on ties), and the workgroup takes the
// pair whose key is the (i+1)-th largest, i its own pair index: with one
// pair per lane by counting larger keys over lane exchanges, else by
// bisection on the key value with wave-wide counts (each lane holds up to
// kRankPerLane pairs).  Every workgroup finds the same order, so this
// permutes the pairs: every work item is still covered once.
constexpr int kRankPerLane = 16;  // == kMaxRankPairs / 64 in tv_plan.h

__device__ __forceinline__ void longest_first(const AttnArgs& a, int bid, WorkItem& it) {
  const int lane = threadIdx.x & 63;
  const int L = kXcds / a.Hkv, per_b = a.S / L, npairs = a.B * per_b;
  const int x = bid % kXcds, target = (bid / kXcds) / a.nRB, ln = x / a.Hkv;
  const int cap = a.tail ? a.Lmax - a.N : a.Lmax;
  int key[kRankPerLane];
#pragma unroll
  for (int k = 0; k < kRankPerLane; ++k) {
    const int p = lane + 64 * k;
    key[k] = -1;
    if (p < npairs) {
      const int pb = p / per_b;
      const int ps = ((ln - pb) % L + L) % L + L * (p % per_b);
      int kvl = a.kv_len ? a.kv_len[pb] : cap;
      kvl = kvl < 0 ? 0 : (kvl > cap ? cap : kvl);
      const int tiles = (kvl + kKeyTile - 1) / kKeyTile + (a.N - 1) / kKeyTile + 1;
      const int work = max(0, min(a.chunk, tiles - ps * a.chunk));  // < 2^14 (plan)
      key[k] = (work << 16) | (0xFFFF - p);
    }
  }
  int p;
  const int nk = (npairs + 63) / 64;  // pair slots in use per lane
  if (nk == 1) {
    // one pair per lane: every lane counts the larger keys by lane exchanges
    int rank = 0;
    for (int q = 0; q < 64; ++q) rank += __shfl(key[0], q) > key[0];
    const unsigned long long hit = __ballot(lane < npairs && rank == target);
    p = __builtin_amdgcn_readfirstlane(hit ? (int)__builtin_ctzll(hit) : 0);
  } else {
    // the largest v with at least target + 1 keys >= v is the wanted key
    int lo = 0, hi = 1 << 30;
    while (hi - lo > 1) {
      const int mid = lo + ((hi - lo) >> 1);
      int c = 0;
#pragma unroll
      for (int k = 0; k < kRankPerLane; ++k)
        if (k < nk) c += __popcll(__ballot(key[k] >= mid));
      if (c >= target + 1) lo = mid;
      else hi = mid;
    }
    p = 0xFFFF - (lo & 0xFFFF);
  }
  it.b = p / per_b;
  it.s = ((ln - it.b) % L + L) % L + L * (p % per_b);
}

// Four output values, or four NaN when the sequence's tree is invalid (the
// NaN is written as a bit pattern: the kernels assume no NaN arithmetic).
__device__ __forceinline__ void store_out4(__bf16* p, const f32x4& acc, float inv, bool nan) {
  const bf16x4 v = {(__bf16)(acc[0] * inv), (__bf16)(acc[1] * inv), (__bf16)(acc[2] * inv),
                    (__bf16)(acc[3] * inv)};
  i16x4 bits = __builtin_bit_cast(i16x4, v);
  if (nan) bits = i16x4{0x7FC0, 0x7FC0, 0x7FC0, 0x7FC0};
  *reinterpret_cast<i16x4*>(p) = bits;
}

// Split-KV partials cross workgroups (and XCDs) through device-scope
// accesses: the sc1 bit makes a store complete only once it is visible at
// device scope and a load read at that level, which is how the compiler
// lowers relaxed agent-scope atomic loads and stores; these are their
// 8- and 16-byte forms.  Publishing then needs only vmcnt(0) before the
// arrival counter, where a release fence would write back the whole L2,
// and the merging workgroup needs no L2 invalidate (which would evict the
// keys that other workgroups are still reading).
__device__ __forceinline__ void store_dev(f32x4* p, f32x4 v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ void store_dev(float2* p, float2 v) {
  asm volatile("global_store_dwordx2 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");
}
__device__ __forceinline__ f32x4 load_dev(const f32x4* p) {
  f32x4 v;
  asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ float2 load_dev(const float2* p) {
  float2 v;
  asm volatile("global_load_dwordx2 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// Plain 16- and 4-byte loads issued as inline assembly, for the prologue:
// the compiler does not track them, so it inserts no wait of its own that
// would also drain the tile DMAs issued after them.  Loads return in issue
// order, so an explicit vmcnt that leaves exactly the younger DMAs
// outstanding covers them; `loaded` then ties each value to that wait.
__device__ __forceinline__ bf16x8 load_b128(const __bf16* p) {
  bf16x8 v;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ int load_i32(const int32_t* p) {
  int v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
// Waits for every outstanding vector memory access; `loaded` values of
// load_dev are tied to the wait so no use is scheduled before it.
__device__ __forceinline__ void wait_all_vm() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
template <class T>
__device__ __forceinline__ void loaded(T& v) {
  asm volatile("" : "+v"(v));
}

__device__ __forceinline__ float wave_max_across_groups(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

// 16 bytes per lane from global memory straight into LDS: lane i reads
// sbase + voff (sbase wave-uniform, voff a per-lane byte offset) and its
// bytes land at lds_addr + 16 * i (lds_addr wave-uniform).  Issued as inline
// assembly so the compiler does not serialise every later LDS read behind
// it; completion is awaited with explicit vmcnt waits.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(sbase)
               : "memory");
}

// A wave-uniform pointer the compiler cannot prove uniform, moved to SGPRs
// (the DMA's base address operand must be scalar).
__device__ __forceinline__ const char* uniform_ptr(const char* p) {
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const char*)(((uint64_t)hi << 32) | lo);
}

// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding).
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// s_waitcnt vmcnt(n) for a wave-uniform n in 0..63 (the prologue's waits:
// queries and DMAs still in flight); anything else waits for everything.
__device__ __forceinline__ void wait_vm_any(int n) {
  switch (n) {
#define TV_WAIT_CASE(k) \
  case k:               \
    wait_vm<k>();       \
    break;
#define TV_WAIT_CASES8(k)                                                                    \
  TV_WAIT_CASE(k) TV_WAIT_CASE(k + 1) TV_WAIT_CASE(k + 2) TV_WAIT_CASE(k + 3) TV_WAIT_CASE(k + 4) \
      TV_WAIT_CASE(k + 5) TV_WAIT_CASE(k + 6) TV_WAIT_CASE(k + 7)
    TV_WAIT_CASES8(0) TV_WAIT_CASES8(8) TV_WAIT_CASES8(16) TV_WAIT_CASES8(24)
    TV_WAIT_CASES8(32) TV_WAIT_CASES8(40) TV_WAIT_CASES8(48) TV_WAIT_CASES8(56)
#undef TV_WAIT_CASES8
#undef TV_WAIT_CASE
    default: wait_vm<0>(); break;
  }
}

// n is (tiles still in flight) x (DMAs per tile); only these values occur
__device__ __forceinline__ void wait_vm_dyn(int n) {
  switch (n) {
    case 1: wait_vm<1>(); break;
    case 2: wait_vm<2>(); break;
    case 3: wait_vm<3>(); break;
    case 4: wait_vm<4>(); break;
    case 6: wait_vm<6>(); break;
    case 8: wait_vm<8>(); break;
    case 12: wait_vm<12>(); break;
    case 16: wait_vm<16>(); break;
    case 24: wait_vm<24>(); break;
    case 32: wait_vm<32>(); break;
    case 48: wait_vm<48>(); break;
    default: wait_vm<0>(); break;
  }
}

// Layout of one 32-key tile in LDS: row-major, D bf16 per row, 16-byte
// chunks XOR-swizzled by the row.  With reads served 256 bytes at a time
// (64 banks; 16 lanes of a ds_read_b128, 32 of a ds_read_b64_tr_b16) the
// swizzle is free of bank conflicts: 16 rows at one logical chunk (the K
// operand reads) land in 16 bank groups, and the transposing V reads (rows
// 8k..8k+7, two adjacent chunks) cover every bank once.  The hardware
// serves the K reads 128 bytes at a time (8 lanes), where rows r and r + 4
// collide: the K reads are 2-way, a third of the LDS-active cycles, as the
// bank-conflict counter shows.  A swizzle free of conflicts at both widths
// (((r & 3) << 1) | ((r >> 2) & 1) | (((r >> 2) ^ (r >> 3)) & 1) << 3 for
// D = 128) removed them and a third of the LDS-active cycles but not a
// cycle of the kernel (about 1% slower), so this one stays.
template <int D>
struct TileLayout {
  static constexpr int kRowBytes = 2 * D;
  static constexpr int kCPR = D / 8;               // 16-byte chunks per row
  static constexpr int kBytes = kKeyTile * kRowBytes;
  static constexpr int kDma = kBytes / 1024;       // 1 KB DMA instructions per tile
  static constexpr int kRowsPerDma = 64 / kCPR;
  __device__ static __forceinline__ int swz(int r) {
    return D == 128 ? (((r & 7) << 1) | ((r >> 3) & 1))
                    : ((((r >> 1) & 3) << 1) | ((r >> 3) & 1));
  }
  __device__ static __forceinline__ int off(int r, int chunk) {
    return r * kRowBytes + ((chunk ^ swz(r)) << 4);
  }
};

// Where a wave's K/V rows come from: the cache of one (sequence, KV head)
// pair, then its tree K/V.  The cache is either padded (row t at kcache +
// t * row_bytes) or paged (row t in pool block btab[t >> shift], whose rows
// are 2^shift apart from kcache + block * 2^shift * row_bytes; a 32-key
// tile never straddles blocks since blocks hold a power of two >= 32 rows).
// Block numbers are clamped into the pool.  Pointers are byte pointers.
struct TreeSrc {
  const char* kcache;
  const char* vcache;
  const char* ktree;
  const char* vtree;
  const int32_t* btab;  // this sequence's block table row, or NULL
  int shift, nblk;      // log2(block size), blocks in the pool
  int row_bytes;  // bytes between consecutive keys
  int rows;       // valid cache rows (the tree's too in the tree-tail layout)
  int nct;        // cache tiles
  int i_hi;       // last tree node the row block can see
};

// Issue this lane's DMA instructions for tile t into the stage at kdst (K
// tile, then V tile).  The scalar base is the tile's first row; rows past
// the valid range are clamped onto a valid row (the mask gives them zero
// weight, the clamp keeps reads in range).  dma_off is the per-lane byte
// offset of its chunk within a full tile.
template <int D, int PW, bool kPaged>
__device__ __forceinline__ void issue_tile(const TreeSrc& src, const uint32_t (&dma_off)[PW],
                                           int wr, int lane, int t, uint32_t kdst) {
  using TL = TileLayout<D>;
  const bool cache = t < src.nct;
  const int first = cache ? t * kKeyTile : (t - src.nct) * kKeyTile;
  const char* kb;
  const char* vb;
  if constexpr (kPaged) {
    size_t tofs = (size_t)first * src.row_bytes;
    if (cache) {
      // A scalar load through the constant address space (the table is
      // read-only here and the tile index wave-uniform): a vector load
      // would make the compiler wait for every DMA in flight.
      typedef const __attribute__((address_space(4))) int32_t ctab_t;
      int blk = ((ctab_t*)src.btab)[__builtin_amdgcn_readfirstlane(first >> src.shift)];
      blk = blk < 0 ? 0 : (blk >= src.nblk ? src.nblk - 1 : blk);
      tofs = (((size_t)blk << src.shift) + (first & ((1 << src.shift) - 1))) * src.row_bytes;
    }
    kb = uniform_ptr((cache ? src.kcache : src.ktree) + tofs);
    vb = uniform_ptr((cache ? src.vcache : src.vtree) + tofs);
  } else {
    kb = (cache ? src.kcache : src.ktree) + (size_t)first * src.row_bytes;
    vb = (cache ? src.vcache : src.vtree) + (size_t)first * src.row_bytes;
  }
  if (cache && (t + 1) * kKeyTile <= src.rows) {
#pragma unroll
    for (int k = 0; k < PW; ++k) {
      const int q = wr * PW + k;
      const bool isv = q >= TL::kDma;
      dma16(isv ? vb : kb, dma_off[k], kdst + (isv ? TL::kBytes : 0) + (q % TL::kDma) * 1024);
    }
    return;
  }
  const int last = cache ? src.rows - 1 : src.i_hi;  // >= first for every existing tile
#pragma unroll
  for (int k = 0; k < PW; ++k) {
    const int q = wr * PW + k;
    const bool isv = q >= TL::kDma;
    const int r = (q % TL::kDma) * TL::kRowsPerDma + lane / TL::kCPR;
    const int row = min(first + r, last) - first;
    const uint32_t off = (uint32_t)(row * src.row_bytes + ((lane % TL::kCPR) ^ TL::swz(r)) * 16);
    dma16(isv ? vb : kb, off, kdst + (isv ? TL::kBytes : 0) + (q % TL::kDma) * 1024);
  }
}

// Where a tile's scores need masking: the cache tail and the tree tiles.
struct MaskInfo {
  int t, nct, kvl, ntt, g4, tail;
  const uint32_t* anc;
};

constexpr float kSlack = 8.f;  // log2 units a row's reference may lag its maximum

// Steps of one 32-key tile for a wave's 32 rows (two 16-row tiles nt).
//
// scores: S^T = K Q^T on the matrix cores; lane (g4, l16) holds
//   S^T[key 16*tt + 4*g4 + j][row 16*nt + l16].
template <int D, int NT>
__device__ __forceinline__ void tile_scores(const unsigned char* kt_lds, const bf16x8 (&qf)[NT][D / 32],
                                            f32x4 (&sc)[2][NT], int g4, int l16) {
  using TL = TileLayout<D>;
  constexpr int NC = D / 32;
  bf16x8 kf[2][NC];
#pragma unroll
  for (int tt = 0; tt < 2; ++tt)
#pragma unroll
    for (int cc = 0; cc < NC; ++cc)
      kf[tt][cc] = *reinterpret_cast<const bf16x8*>(kt_lds + TL::off(16 * tt + l16, 4 * cc + g4));
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < NC; ++cc)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[tt][cc], qf[nt][cc], acc, 0, 0, 0);
      sc[tt][nt] = acc;
    }
}

// mask: -inf for cache keys at or past kv_len and for tree keys outside
// the row's ancestor-or-self set (one 32-bit word of its bitmask per tile).
template <int NT>
__device__ __forceinline__ void tile_mask(f32x4 (&sc)[2][NT], const MaskInfo& mk,
                                          const int (&node_rel)[NT]) {
  if (mk.tail) {
    // Tree-tail layout: key k of the tile is node s + k (s < 0: a context
    // row).  Its visibility bits are a 32-bit window of the row's ancestor
    // bitmask, words w0 and w0 + 1, with all-ones standing in for context
    // rows (word -1) and zeros past the last word.
    const int s = mk.t * kKeyTile - mk.kvl;  // > -kKeyTile in the masked tiles
    const int w0 = s >> 5, sh = s & 31;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint32_t* wp = mk.anc + node_rel[nt] * mk.ntt;
      const uint32_t lo = w0 < 0 ? 0xFFFFFFFFu : wp[w0];
      const uint32_t hi = w0 + 1 < mk.ntt ? wp[w0 + 1] : 0u;
      const uint32_t bits = (uint32_t)((((uint64_t)hi << 32) | lo) >> sh);
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (!((bits >> (16 * tt + 4 * mk.g4 + j)) & 1u)) sc[tt][nt][j] = -INFINITY;
    }
  } else if (mk.t < mk.nct) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool vis = mk.t * kKeyTile + 16 * tt + 4 * mk.g4 + j < mk.kvl;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          if (!vis) sc[tt][nt][j] = -INFINITY;
      }
  } else {
    const int word = mk.t - mk.nct;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint32_t bits = mk.anc[node_rel[nt] * mk.ntt + word];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (!((bits >> (16 * tt + 4 * mk.g4 + j)) & 1u)) sc[tt][nt][j] = -INFINITY;
    }
  }
}

// reference: online softmax in base 2 with a lazily moved reference.  A
//   row's reference m (log2 units) only moves when one of its scores
//   exceeds it by more than kSlack, so weights stay below 2^kSlack (far
//   inside the fp32 and bf16 ranges) and rescaling is rare.  Each lane
//   compares its raw scores with thr = (m + kSlack) / c; only a moving tile
//   pays for exact row maxima, and rows that move rescale O and l.
template <int DT, int NT>
__device__ __forceinline__ void tile_reference(const f32x4 (&sc)[2][NT], float (&m)[NT],
                                               float (&thr)[NT], f32x4 (&o)[DT][NT],
                                               f32x4 (&lacc)[NT], float c, float inv_c) {
  float mx[NT];
  bool move = false;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float v = fmaxf(fmaxf(sc[0][nt][0], sc[0][nt][1]), sc[0][nt][2]);
    v = fmaxf(fmaxf(v, sc[0][nt][3]), sc[1][nt][0]);
    v = fmaxf(fmaxf(v, sc[1][nt][1]), sc[1][nt][2]);
    v = fmaxf(v, sc[1][nt][3]);
    mx[nt] = v;
    move |= v > thr[nt];
  }
  if (__any(move)) {
    // rare: a row that has not moved keeps its scale; its m may still be -inf
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      mx[nt] = wave_max_across_groups(mx[nt]) * c;
      const bool moved = mx[nt] > m[nt] + kSlack;
      const float alpha = moved ? __builtin_amdgcn_exp2f(m[nt] - mx[nt]) : 1.f;
      m[nt] = moved ? mx[nt] : m[nt];
      thr[nt] = (m[nt] + kSlack) * inv_c;
      lacc[nt] *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt][nt] *= alpha;
    }
  }
}

// weights: the bf16 P^T operand, exactly as it lies in the accumulators.
template <int NT>
__device__ __forceinline__ void tile_weights(const f32x4 (&sc)[2][NT], const float (&m)[NT], float c,
                                             bf16x8 (&pf)[NT]) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float mref = fmaxf(m[nt], -3.0e38f);  // rows with nothing visible yet: weights 0
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        pf[nt][4 * tt + j] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sc[tt][nt][j], c, -mref));
  }
}

// values: row sums ones^T P^T into lacc (same rounded weights as the
//   numerator) and O^T += V^T P^T with V^T from transposing LDS reads: lane
//   (g4, l16) receives V[key 4*g4 + j (+16)][16*dt + l16], the key order of P^T.
template <int D, int NT>
__device__ __forceinline__ void tile_values(const unsigned char* vt_lds, const bf16x8 (&pf)[NT],
                                            const bf16x8& ones, f32x4 (&o)[D / 16][NT],
                                            f32x4 (&lacc)[NT], int g4, int l16) {
  using TL = TileLayout<D>;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
    lacc[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[nt], lacc[nt], 0, 0, 0);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const int rr = 4 * g4 + (l16 >> 2);
    const int chunk = 2 * dt + ((l16 & 3) >> 1);
    const int inb = 8 * (l16 & 1);
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(vt_lds + TL::off(rr, chunk) + inb));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(vt_lds + TL::off(rr + 16, chunk) + inb));
    const bf16x4 lob = __builtin_bit_cast(bf16x4, lo), hib = __builtin_bit_cast(bf16x4, hi);
    const bf16x8 vf = {lob[0], lob[1], lob[2], lob[3], hib[0], hib[1], hib[2], hib[3]};
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      o[dt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[nt], o[dt][nt], 0, 0, 0);
  }
}

// The whole tile in order (the loop form without lookahead).
template <int D, int NT, bool kMasked>
__device__ __forceinline__ void attend_tile(const unsigned char* kt_lds, const bf16x8 (&qf)[NT][D / 32],
                                            f32x4 (&o)[D / 16][NT], f32x4 (&lacc)[NT],
                                            float (&m)[NT], float (&thr)[NT], const bf16x8& ones,
                                            float c, float inv_c, const MaskInfo& mk,
                                            const int (&node_rel)[NT], int g4, int l16) {
  f32x4 sc[2][NT];
  // The score products run at raised wave priority: the SIMD's other wave
  // is then mostly in its softmax (vector work) while these matrix
  // instructions issue back to back (measured 5-8% faster on matrix-bound
  // shapes than equal priority or raising it for the value products too).
  __builtin_amdgcn_s_setprio(1);
  tile_scores<D, NT>(kt_lds, qf, sc, g4, l16);
  __builtin_amdgcn_s_setprio(0);
  if (kMasked) tile_mask<NT>(sc, mk, node_rel);
  tile_reference<D / 16, NT>(sc, m, thr, o, lacc, c, inv_c);
  bf16x8 pf[NT];
  tile_weights<NT>(sc, m, c, pf);
  tile_values<D, NT>(kt_lds + TileLayout<D>::kBytes, pf, ones, o, lacc, g4, l16);
}

// Merge of the chunk partials of one row block, run by the workgroup whose
// chunk arrived last: out = sum_s e_s O_s / sum_s e_s l_s, e_s = 2^(m_s - m*),
// folded in online over s in batches of loads.  Wave w takes one 16-row
// tile and every WPN-th 16-column tile of it (or several row tiles when the
// block has more row tiles than the workgroup has waves), so each lane
// reads its rows' (m, l) once.
template <int D, int RB, int kWaves>
__device__ __forceinline__ void merge_chunks(const AttnArgs& a, size_t part0, int nval, int b,
                                             int g, int r0, bool bad, int wave, int lane) {
  constexpr int DT = D / 16, NTG = RB / 16;
  constexpr bool kSplitCols = kWaves >= NTG;
  constexpr int WPN = kSplitCols ? kWaves / NTG : 1;  // waves per row tile
  constexpr int NPW = kSplitCols ? 1 : NTG / kWaves;  // row tiles per wave
  constexpr int DPW = DT / WPN;                       // column tiles per wave
  constexpr int UB = 32 / DPW;                        // chunks per batch of loads
  // every wave gets whole column tiles of one row tile, or whole row tiles
  static_assert(kSplitCols ? (kWaves % NTG == 0 && DT % WPN == 0) : (NTG % kWaves == 0),
                "merge split");
  const int g4 = lane >> 4, l16 = lane & 15;
#pragma unroll
  for (int k = 0; k < NPW; ++k) {
    const int ntg = kSplitCols ? wave % NTG : wave + k * kWaves;
    const int dt0 = kSplitCols ? wave / NTG : 0;
    const int row = ntg * 16 + l16;
    float m = -INFINITY, l = 0.f;
    f32x4 acc[DPW];
#pragma unroll
    for (int j = 0; j < DPW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < nval; s0 += UB) {
      float2 ml[UB];
      f32x4 ov[UB][DPW];
#pragma unroll
      for (int u = 0; u < UB; ++u)
        if (s0 + u < nval) {
          const size_t ps = part0 + s0 + u;
          ml[u] = load_dev(&a.ws_ml[ps * RB + row]);
#pragma unroll
          for (int j = 0; j < DPW; ++j)
            ov[u][j] = load_dev(&a.ws_o[(ps * DT * NTG + (dt0 + j * WPN) * NTG + ntg) * 64 + lane]);
        }
      wait_all_vm();
#pragma unroll
      for (int u = 0; u < UB; ++u)
        if (s0 + u < nval) {
          loaded(ml[u]);
#pragma unroll
          for (int j = 0; j < DPW; ++j) loaded(ov[u][j]);
        }
#pragma unroll
      for (int u = 0; u < UB; ++u)
        if (s0 + u < nval && ml[u].x != -INFINITY) {
          const float mn = fmaxf(m, ml[u].x);
          const float ea = __builtin_amdgcn_exp2f(m - mn);  // 0 while m = -inf
          const float eb = __builtin_amdgcn_exp2f(ml[u].x - mn);
          l = l * ea + eb * ml[u].y;
#pragma unroll
          for (int j = 0; j < DPW; ++j) acc[j] = acc[j] * ea + eb * ov[u][j];
          m = mn;
        }
    }
    const int r = r0 + row;
    if (r < a.M) {
      const int node = r / a.G, h = g * a.G + r % a.G;
      __bf16* op = a.out + ((size_t)(b * a.N + node) * a.Hq + h) * D + 4 * g4;
      const float inv = 1.f / l;
#pragma unroll
      for (int j = 0; j < DPW; ++j) store_out4(op + 16 * (dt0 + j * WPN), acc[j], inv, bad);
    }
  }
}

// A workgroup of WR x WK wave64s: WR row groups x WK key groups.  A wave owns 32 rows of its row group; the WR
// waves of a key group share one LDS ring and walk that group's tiles (every
// WK-th tile of the chunk) in lock step; WK > 1 groups merge their partial
// softmax states in LDS at the end.
template <int D, int WR, int WK, int NS, bool kPaged, bool kShareQ>
__global__ __launch_bounds__(64 * WR * WK) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_main(AttnArgs a) {
  using TL = TileLayout<D>;
  constexpr int kThreads = 64 * WR * WK;
  constexpr int kWaves = WR * WK;
  constexpr int RB = kRowsPerWave * WR; // rows per workgroup
  constexpr int NT = kRowsPerWave / 16; // 16-row tiles per wave
  constexpr int NTG = RB / 16;          // 16-row tiles per workgroup
  constexpr int NC = D / 32;            // 32-wide head-dim chunks (QK^T)
  constexpr int DT = D / 16;            // 16-wide head-dim tiles (PV)
  constexpr int STAGE = 2 * TL::kBytes; // K tile + V tile
  constexpr int PW = 2 * TL::kDma / WR; // DMAs per wave per tile
  static_assert(PW >= 1 && PW * WR == 2 * TL::kDma, "DMA split");
  static_assert(NS >= 1, "ring does not fit");
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  WorkItem it{};
  if (!work_item(gridDim.x, a.nwork, a.S, a.nRB, a.spread, a.B, a.Hkv, blockIdx.x, it)) return;
  if (a.spread == 2) longest_first(a, blockIdx.x, it);
  const int s = it.s, rb = it.rb, g = it.g, b = it.b;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave % WR, wk = wave / WR;
  const int g4 = lane >> 4, l16 = lane & 15;

  const int r0 = rb * RB;
  const int rows = min(RB, a.M - r0);
  const int i_lo = r0 / a.G, i_hi = (r0 + rows - 1) / a.G;
  const Segment sg = segment(a, b, i_hi);
  const int kvl = sg.kvl, nct = sg.nct, T = sg.T;
  const int ntt = i_hi / kKeyTile + 1;  // words of a node's ancestor bitmask
  const int t0 = s * a.chunk;
  const int t1 = min(T, t0 + a.chunk);
  if (t0 >= t1) return;  // empty chunk: the merge reads only chunks with tiles
  const bool has_tree = a.tail ? t1 * kKeyTile > kvl : t1 > nct;

  constexpr int RING = WK * NS * STAGE;
  const uint32_t ring = (uint32_t)(uintptr_t)smem + wk * NS * STAGE;
  const unsigned char* ring_ptr = smem + wk * NS * STAGE;
  // the block's queries (kShareQ) follow the rings, then the tree tables
  static_assert(!kShareQ || (WK > 1 && WR > 1), "queries are shared between key groups");
  constexpr bool qshare = kShareQ;
  const bool qload = !qshare || wk == 0;  // this wave loads its queries from memory
  unsigned char* qlds = smem + RING;
  uint32_t* anc = reinterpret_cast<uint32_t*>(smem + RING + (qshare ? RB * D * 2 : 0));
  const int anc_nodes = RB / a.G + 2;
  int32_t* par = reinterpret_cast<int32_t*>(anc + anc_nodes * ntt);
  int* flag = par + a.N;

  const size_t krow = (size_t)a.Hkv * D;  // elements between consecutive keys
  const size_t cache0 = kPaged ? 0 : (size_t)(b / a.cgroup) * a.Lmax * krow;  // paged: pool
  const __bf16* kcache = a.kc + cache0 + (size_t)g * D;
  const __bf16* vcache = a.vc + cache0 + (size_t)g * D;
  const size_t tree0 = (size_t)b * a.N * krow + (size_t)g * D;  // unused with a tree tail
  const __bf16* ktree = a.tail ? kcache : a.kt + tree0;
  const __bf16* vtree = a.tail ? vcache : a.vt + tree0;

  // This lane's share of the DMA instructions of one tile: instruction q
  // (q < kDma: K, else V) covers tile rows j*kRowsPerDma.. (j = q % kDma);
  // lane i fetches row j*kRowsPerDma + i/kCPR at the logical chunk that the
  // swizzle places at physical chunk i % kCPR.  dma_off is that byte offset
  // from the first row of a full tile.
  uint32_t dma_off[PW];
#pragma unroll
  for (int k = 0; k < PW; ++k) {
    const int q = wr * PW + k;
    const int r = (q % TL::kDma) * TL::kRowsPerDma + lane / TL::kCPR;
    dma_off[k] = (uint32_t)(r * (int)krow * 2 + ((lane % TL::kCPR) ^ TL::swz(r)) * 16);
  }
  const TreeSrc src{(const char*)kcache,
                    (const char*)vcache,
                    (const char*)ktree,
                    (const char*)vtree,
                    kPaged ? a.block_table + (size_t)b * a.max_blocks : nullptr,
                    a.block_shift,
                    a.num_blocks,
                    (int)krow * 2,
                    a.tail ? kvl + i_hi + 1 : kvl,
                    nct,
                    i_hi};

  // iteration i handles tile t0 + wk + WK*i of this wave's key group; all
  // waves run n_iter iterations so the per-iteration barriers line up
  const int n_iter = t1 > t0 ? (t1 - t0 + WK - 1) / WK : 0;
  const int n_mine = t0 + wk < t1 ? (t1 - t0 - wk + WK - 1) / WK : 0;  // valid tiles

  // Issue order: parents, queries, then the first tiles' DMAs, all before
  // any of them is used.  When the WR waves of a key group share its ring
  // (WR > 1) the prologue fills every stage: the ring's own refills come
  // after a workgroup barrier, and the first of them would otherwise wait
  // for the first tile's round trip.  A single-wave key group refills
  // before its waits and keeps one stage for that.  (Measured on the
  // Qwen3-8B-shaped 64-node, 4096-row call, together with the shared
  // queries below: 20.6 -> 19.6 us.)
  constexpr int kParPerThread = (kMaxNodes + kThreads - 1) / kThreads;
  constexpr int NQ = NT * NC;  // query loads per lane
  constexpr int kPro = WR > 1 ? NS : NS - 1;
  const int npro = min(kPro, n_mine);  // tiles the prologue issues
  int pv[kParPerThread];
  if (has_tree) {
    // indices clamped rather than branched on, so the loads stay in flight
    const int32_t* pr = a.parent + (size_t)b * a.N;
#pragma unroll
    for (int k = 0; k < kParPerThread; ++k) {
      const int i = tid + kThreads * k;
      pv[k] = a.parent ? load_i32(pr + (i < a.N ? i : a.N - 1)) : i - 1;  // NULL: a chain
    }
  }

  // ---- queries: B operand of S^T = K Q^T, lane holds Q[row l16][8*g4 .. +8]
  const int wrow0 = r0 + kRowsPerWave * wr;
  bf16x8 qf[NT][NC];
  bool qok[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = wrow0 + nt * 16 + l16;
    const bool ok = r < a.M;
    qok[nt] = ok;
    const int node = ok ? r / a.G : 0;
    const int h = g * a.G + (ok ? r % a.G : 0);
    const __bf16* qp = a.q + ((size_t)(b * a.N + node) * a.Hq + h) * D + 8 * g4;
    if (qload) {
#pragma unroll
      for (int c = 0; c < NC; ++c) qf[nt][c] = load_b128(qp + 32 * c);
    }
  }

#pragma unroll
  for (int i = 0; i < kPro; ++i)
    if (i < n_mine) issue_tile<D, PW, kPaged>(src, dma_off, wr, lane, t0 + wk + WK * i, ring + i * STAGE);

  // ---- tree structure: ancestor-or-self bitmask of this block's nodes
  if (has_tree) {
    // the parents are done once at most the queries and the DMAs are in flight
    wait_vm_any((qload ? NQ : 0) + npro * PW);
#pragma unroll
    for (int k = 0; k < kParPerThread; ++k) loaded(pv[k]);
    int bad = 0;
#pragma unroll
    for (int k = 0; k < kParPerThread; ++k) {
      const int i = tid + kThreads * k;
      if (i >= a.N) break;
      const int p = pv[k];
      par[i] = p;
      bad |= (i == 0) ? (p != -1) : (p < 0 || p >= i);
    }
    bad = __syncthreads_or(bad);
    const int nodes = i_hi - i_lo + 1;
    for (int t = tid; t < nodes; t += kThreads) {
      uint32_t* wd = anc + t * ntt;
      for (int k = 0; k < ntt; ++k) wd[k] = 0u;
      int u = i_lo + t;
      for (;;) {
        wd[u >> 5] |= 1u << (u & 31);
        if (u == 0) break;
        const int p = par[u];
        if (p < 0 || p >= u) break;  // invalid tree: the output becomes NaN
        u = p;
      }
    }
    if (tid == 0) *flag = bad;
    __syncthreads();
  }

  // the queries are done once at most the DMAs are in flight; rows past the
  // block's last row get zero queries.  Shared queries sit in LDS in the
  // tile layout, one 32-row tile per row group, read like the K operand.
  if (qload) {
    wait_vm_any(npro * PW);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        loaded(qf[nt][c]);
        if (!qok[nt]) qf[nt][c] = bf16x8{};
      }
  }
  // (the other key groups read them after the first ring step's barrier)
  unsigned char* qt = qlds + wr * TL::kBytes;
  if (qshare && wk == 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        *reinterpret_cast<bf16x8*>(qt + TL::off(16 * nt + l16, 4 * c + g4)) = qf[nt][c];
  }

  // O^T accumulators, and l: row sums of the bf16 weights, accumulated on
  // the matrix cores as ones^T P^T so numerator and denominator see the same
  // rounded weights (all 4 entries of lacc[nt] hold the lane's row sum)
  f32x4 o[DT][NT], lacc[NT];
  float m[NT];
  const bf16x8 ones = {(__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f,
                       (__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m[nt] = -INFINITY;
    lacc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // node of this lane's row in each 16-row tile, relative to i_lo
  int node_rel[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = wrow0 + nt * 16 + l16;
    node_rel[nt] = (r < a.M ? r : a.M - 1) / a.G - i_lo;
  }

  float thr[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) thr[nt] = -INFINITY;  // m = -inf: any visible score moves
  const float inv_c = 1.f / a.c;
  bf16x8 ones_v = ones;
  asm volatile("" : "+v"(ones_v));  // keep it in registers, not rebuilt every tile
  // Ring step of iteration i: wait for this key group's tile i and refill
  // the ring.  With WR > 1 the prologue issued tiles 0..NS-1 and step j >= 1
  // issues tile j+NS-1, so my DMAs of tile i are done once at most
  // min(later tiles, NS-1 at step 0, NS-2 after) tiles' DMAs are
  // outstanding; the barrier makes the whole group's visible and guarantees
  // the slot of tile i-1 is no longer read.
  auto ring_step = [&](int i) {
    const bool mine = i < n_mine;
    if (WR > 1) {
      if (mine) wait_vm_dyn(min(n_mine - 1 - i, i == 0 ? NS - 1 : NS - 2) * PW);
      __syncthreads();
      if (i >= 1 && i + NS - 1 < n_mine)
        issue_tile<D, PW, kPaged>(src, dma_off, wr, lane, t0 + wk + WK * (i + NS - 1),
                          ring + ((i + NS - 1) % NS) * STAGE);
    } else {
      if (i + NS - 1 < n_mine)
        issue_tile<D, PW, kPaged>(src, dma_off, wr, lane, t0 + wk + WK * (i + NS - 1),
                          ring + ((i + NS - 1) % NS) * STAGE);
      if (mine) wait_vm_dyn(min(n_mine - 1 - i, NS - 1) * PW);
    }
  };
  // Full cache tiles first, without masking; the tiles that need a mask
  // (the cache tail, then the tree tiles) all come after them.  Shared
  // queries are read behind the first step's workgroup barrier: every
  // workgroup here has n_iter >= 1, so this loop always runs step 0.
  auto shared_queries = [&]() {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        qf[nt][c] = *reinterpret_cast<const bf16x8*>(qt + TL::off(16 * nt + l16, 4 * c + g4));
  };
  int i = 0;
  for (; i < n_iter; ++i) {
    ring_step(i);
    if (i == 0 && qshare && wk != 0) shared_queries();
    const int t = t0 + wk + WK * i;
    if (i >= n_mine || t >= nct || (t + 1) * kKeyTile > kvl) break;
    const MaskInfo mk{t, nct, kvl, ntt, g4, a.tail, anc};
    attend_tile<D, NT, false>(ring_ptr + (i % NS) * STAGE, qf, o, lacc, m, thr, ones_v, a.c, inv_c,
                              mk, node_rel, g4, l16);
  }
  for (bool stepped = true; i < n_iter; ++i, stepped = false) {
    if (!stepped) ring_step(i);
    if (i >= n_mine) continue;
    const int t = t0 + wk + WK * i;
    const MaskInfo mk{t, nct, kvl, ntt, g4, a.tail, anc};
    attend_tile<D, NT, true>(ring_ptr + (i % NS) * STAGE, qf, o, lacc, m, thr, ones_v, a.c, inv_c,
                             mk, node_rel, g4, l16);
  }

  float lsum[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) lsum[nt] = lacc[nt][0];
  const int invalid = has_tree ? *flag : 0;
  const int bg = b * a.Hkv + g;
  const size_t grp = (size_t)bg * a.nRB + rb;  // row block id
  const size_t part0 = grp * a.S;              // its first chunk partial

  // Final values of one 16x16 fragment (dt, ntg) of this workgroup's rows:
  // either the normalised bf16 output (single chunk) or the chunk partial.
  auto emit = [&](int dt, int ntg, const f32x4& acc, float mstar, float l) {
    const int row = ntg * 16 + l16;
    if (a.S == 1) {
      const int r = r0 + row;
      if (r < a.M) {
        const int node = r / a.G, h = g * a.G + r % a.G;
        store_out4(a.out + ((size_t)(b * a.N + node) * a.Hq + h) * D + 16 * dt + 4 * g4, acc,
                   1.f / l, invalid != 0);
      }
    } else {
      f32x4* po = &a.ws_o[((part0 + s) * DT * NTG + dt * NTG + ntg) * 64 + lane];
      float2* pml = &a.ws_ml[(part0 + s) * RB + row];
      if (a.fused) {  // read by another workgroup of this kernel
        store_dev(po, acc);
        if (dt == 0 && g4 == 0) store_dev(pml, make_float2(mstar, l));
      } else {        // read by the merge kernel
        *po = acc;
        if (dt == 0 && g4 == 0) *pml = make_float2(mstar, l);
      }
    }
  };

  if (WK == 1) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) emit(dt, wr * NT + nt, o[dt][nt], m[nt], lsum[nt]);
  } else {
    // ---- merge the WK key groups of each row group (same rows, disjoint keys)
    __syncthreads();  // rings and tree tables are dead from here on
    f32x4* obuf = reinterpret_cast<f32x4*>(smem);
    float2* mlbuf = reinterpret_cast<float2*>(smem + (size_t)kWaves * kRowsPerWave * D * 4);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) obuf[((wave * DT + dt) * NT + nt) * 64 + lane] = o[dt][nt];
    if (g4 == 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        mlbuf[wave * kRowsPerWave + nt * 16 + l16] = make_float2(m[nt], lsum[nt]);
    }
    __syncthreads();
    for (int f = wk; f < DT * NT; f += WK) {
      const int dt = f / NT, nt = f % NT;
      const int rw = nt * 16 + l16;  // row within the wave's 32
      float mw[WK], mstar = -INFINITY;
#pragma unroll
      for (int k = 0; k < WK; ++k) {
        mw[k] = mlbuf[(k * WR + wr) * kRowsPerWave + rw].x;
        mstar = fmaxf(mstar, mw[k]);
      }
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      float l = 0.f;
#pragma unroll
      for (int k = 0; k < WK; ++k) {
        const float e = mw[k] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw[k] - mstar);
        l += e * mlbuf[(k * WR + wr) * kRowsPerWave + rw].y;
        acc += e * obuf[(((k * WR + wr) * DT + dt) * NT + nt) * 64 + lane];
      }
      emit(dt, wr * NT + nt, acc, mstar, l);
    }
  }
  if (a.S == 1 || !a.fused) return;

  // ---- fused split-KV merge: the chunk that arrives last merges its row
  // block.  Every workgroup publishes its partial (device-scope stores,
  // completed before the count), then counts itself in; the one that
  // completes the count merges and resets the counter for the next call.
  // Only chunks that hold tiles take part: nval of them.
  const int nval = min(a.S, (T + a.chunk - 1) / a.chunk);
  __shared__ int s_last;
  if (has_tree && tid == 0)  // every row block has a chunk with tree tiles
    __hip_atomic_store(a.tree_bad + grp, invalid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  wait_all_vm();
  __syncthreads();
  if (tid == 0) {
    const unsigned int before =
        __hip_atomic_fetch_add(a.arrived + grp, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = before + 1 == (unsigned int)nval;
    if (last) __hip_atomic_store(a.arrived + grp, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = last;
  }
  __syncthreads();
  if (!s_last) return;
  const bool bad = __hip_atomic_load(a.tree_bad + grp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
  merge_chunks<D, RB, kWaves>(a, part0, nval, b, g, r0, bad, wave, lane);
}

// Second kernel of the split-KV plans whose merge is too large for one
// workgroup: out = sum_s e_s O_s / sum_s e_s l_s with e_s = 2^(m_s - m*),
// folded in online over batches of U chunks.  Only chunks that hold tiles
// of this row block were written.  One wave per 16x16 fragment.  The
// parents (for the tree check), kv_len and the first batch of partials are
// all requested before any is used, so a merge of up to U chunks waits for
// one round of memory latency: the first batch reads the slots of the
// first min(S, U) chunks whether or not they were written by this call
// (they lie inside the workspace), and only the nval chunks that hold
// tiles, known once kv_len arrives, are folded in.
template <int D, int RB>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
  constexpr int NTG = RB / 16, DT = D / 16, U = 16;
  constexpr int kParPerThread = kMaxNodes / 256;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  const int F = blockIdx.x * 4 + wave;  // fragment id; all 4 of a block share (b,g,rb)
  const int per_blk = DT * NTG;
  const int blk = F / per_blk, f = F % per_blk;
  const int rb = blk % a.nRB, bg = blk / a.nRB;
  const int b = bg / a.Hkv, g = bg % a.Hkv;
  int pv[kParPerThread];
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = threadIdx.x + 256 * k;
    pv[k] = i >= a.N ? 0 : (a.parent ? a.parent[(size_t)b * a.N + i] : i - 1);
  }
  const int dt = f / NTG, ntg = f % NTG;
  const int row = ntg * 16 + l16, r = rb * RB + row;
  // chunks of this row block that hold tiles (the same count the main
  // kernel derives from kv_len and the block's last node)
  const int i_hi = (min(rb * RB + RB, a.M) - 1) / a.G;
  const size_t base = (size_t)(bg * a.nRB + rb) * a.S;  // first chunk partial
  float2 ml0[U];
  f32x4 ov0[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (u < a.S) {
      ml0[u] = a.ws_ml[(base + u) * RB + row];
      ov0[u] = a.ws_o[((base + u) * DT * NTG + dt * NTG + ntg) * 64 + lane];
    }
  const int T = segment(a, b, i_hi).T;
  const int nval = min(a.S, (T + a.chunk - 1) / a.chunk);
  float m = -INFINITY, l = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nval; s0 += U) {
    float2 ml[U];
    f32x4 ov[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (s0 + u < nval) {
        if (s0 == 0) {
          ml[u] = ml0[u];
          ov[u] = ov0[u];
        } else {
          ml[u] = a.ws_ml[(base + s0 + u) * RB + row];
          ov[u] = a.ws_o[((base + s0 + u) * DT * NTG + dt * NTG + ntg) * 64 + lane];
        }
      }
    float mb = m;
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (s0 + u < nval) mb = fmaxf(mb, ml[u].x);
    if (mb != -INFINITY) {  // else every chunk so far saw no key: nothing to add
      const float ea = __builtin_amdgcn_exp2f(m - mb);  // 0 while m = -inf
      l *= ea;
      acc *= ea;
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (s0 + u < nval && ml[u].x != -INFINITY) {
          const float e = __builtin_amdgcn_exp2f(ml[u].x - mb);
          l += e * ml[u].y;
          acc += e * ov[u];
        }
      m = mb;
    }
  }
  int bad = 0;
#pragma unroll
  for (int k = 0; k < kParPerThread; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < a.N) bad |= (i == 0) ? (pv[k] != -1) : (pv[k] < 0 || pv[k] >= i);
  }
  bad = __syncthreads_or(bad);
  if (r >= a.M) return;
  const int node = r / a.G, h = g * a.G + r % a.G;
  store_out4(a.out + ((size_t)(b * a.N + node) * a.Hq + h) * D + 16 * dt + 4 * g4, acc, 1.f / l,
             bad != 0);
}

template <int D, int WR, int WK, int NS, bool kPaged, bool kShareQ>
static hipError_t launch_main(const AttnArgs& a, const AttnPlan& p, hipStream_t st) {
  hipError_t e = hipFuncSetAttribute((const void*)attn_main<D, WR, WK, NS, kPaged, kShareQ>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)p.lds_bytes);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_main<D, WR, WK, NS, kPaged, kShareQ>), dim3(p.grid), dim3(64 * WR * WK),
                     p.lds_bytes, st, a);
  return hipGetLastError();
}

template <int D, int ARR, bool kPaged>
static hipError_t launch_attn_t(const AttnArgs& a, const AttnPlan& p, hipStream_t st) {
  constexpr Arrangement ar = kArrangements[ARR];
  constexpr int NS = arr_stages(ar, D);
  if constexpr (NS == 0) {
    return hipErrorInvalidValue;  // never planned: the ring does not fit
  } else {
    // query sharing is a separate instantiation, so the kernels without it
    // carry none of its code or scalar registers
    hipError_t e;
    if constexpr (ar.WK > 1 && ar.WR > 1)
      e = p.qshare ? launch_main<D, ar.WR, ar.WK, NS, kPaged, true>(a, p, st)
                   : launch_main<D, ar.WR, ar.WK, NS, kPaged, false>(a, p, st);
    else
      e = launch_main<D, ar.WR, ar.WK, NS, kPaged, false>(a, p, st);
    if (e != hipSuccess || p.S == 1 || p.fused) return e;
    constexpr int RB = kRowsPerWave * ar.WR;
    const int frags = a.B * a.Hkv * p.nRB * (D / 16) * (RB / 16);
    hipLaunchKernelGGL((attn_combine<D, RB>), dim3(frags / 4), dim3(256), 0, st, a);
    return hipGetLastError();
  }
}

template <int D, int K = 0>
static hipError_t launch_attn_d(const AttnArgs& a, const AttnPlan& p, hipStream_t st) {
  if constexpr (K < kNumArrangements) {
    if (p.arr == K)
      return a.block_table ? launch_attn_t<D, K, true>(a, p, st)
                           : launch_attn_t<D, K, false>(a, p, st);
    return launch_attn_d<D, K + 1>(a, p, st);
  } else {
    return hipErrorInvalidValue;
  }
}

hipError_t launch_attention(const void* q, const void* kc, const void* vc, const void* kt,
                            const void* vt, const int32_t* parent, const int32_t* kv_len,
                            void* out, int B, int N, int Hq, int Hkv, int D, int Lmax,
                            float scale, void* ws, const AttnPlan& p, hipStream_t st,
                            const int32_t* block_table, int block_shift, int max_blocks,
                            int num_blocks, int cgroup) {
  AttnArgs a;
  a.tail = kt == nullptr;
  a.cgroup = cgroup;
  a.block_table = block_table;
  a.block_shift = block_shift;
  a.max_blocks = max_blocks;
  a.num_blocks = num_blocks;
  a.q = (const __bf16*)q;
  a.kc = (const __bf16*)kc;
  a.vc = (const __bf16*)vc;
  a.kt = (const __bf16*)kt;
  a.vt = (const __bf16*)vt;
  a.parent = parent;
  a.kv_len = kv_len;
  a.out = (__bf16*)out;
  a.arrived = (unsigned int*)ws;
  a.tree_bad = (int*)ws + kSyncGroups;
  a.ws_o = (f32x4*)((char*)ws + p.ws_sync_bytes);
  a.ws_ml = (float2*)((char*)ws + p.ws_sync_bytes + p.ws_o_bytes);
  a.B = B;
  a.N = N;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Lmax = Lmax;
  a.G = p.G;
  a.M = p.M;
  a.nRB = p.nRB;
  a.S = p.S;
  a.chunk = p.chunk;
  a.nwork = p.nwork;
  a.fused = p.fused;
  a.spread = p.spread;
  a.c = scale * 1.4426950408889634f;
  return D == 128 ? launch_attn_d<128>(a, p, st) : launch_attn_d<64>(a, p, st);
}

}  // namespace tv
