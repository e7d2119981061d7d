// Host-side launch planning shared by the entry points and the kernels'
// launchers.  Pure C++ (no HIP): the plans depend only on host-known sizes.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace tv {

constexpr int kKeyTile = 32;       // keys one wave consumes per step
constexpr int kXcds = 8;           // MI355X accelerator complex dies
constexpr int kMaxRankPairs = 1024;  // longest-first ranking: pairs per XCD lane (16 per lane)
constexpr int kMaxNodes = 2048;    // == TV_MAX_NODES

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Attention work decomposition.  Rows of one (sequence, KV head) pair are the
// N*G (node, query-head-in-group) pairs, row r = node * G + head_in_group.
// A workgroup takes a block of RB = 32*WR consecutive rows and one
// fixed-size chunk of the key tiles (cache tiles first, then tree tiles).
// Its WR*WK waves form WR row groups (32 rows per wave) times WK key groups
// that split the chunk's tiles between them; each key group streams its
// tiles through an LDS ring of NS stages.  Arrangements are sized so that a
// CU holds 8 waves (two per SIMD), from one or more workgroups.
constexpr int kRowsPerWave = 32;
// Split-KV plans keep per-row-block sync words (arrival counter, tree flag)
// in a fixed region at the start of the workspace, the same place for every
// shape, so that one zero-filled workspace can serve calls of any sizes: a
// call's partials never overlap another call's counters, and each call
// leaves its counters at zero.  Plans with more row blocks do not split.
constexpr int kSyncGroups = 4096;
constexpr size_t kSyncBytes = (size_t)kSyncGroups * 8;
constexpr int kFusedMergeBytes = 1024;
constexpr int kWavesPerCU = 8;
constexpr size_t kMaxLds = 160 * 1024;

struct Arrangement {
  int WR, WK, NS128, NS64;
};
// WR x WK waves; ring stages for D = 128 and D = 64 (16 KB / 8 KB stages)
constexpr Arrangement kArrangements[] = {
    {8, 1, 4, 4}, {4, 2, 4, 4}, {2, 4, 2, 4}, {1, 8, 0, 2},
    {4, 1, 4, 4}, {2, 2, 2, 4}, {2, 1, 2, 4},
};
constexpr int kNumArrangements = sizeof(kArrangements) / sizeof(kArrangements[0]);

constexpr int arr_stages(const Arrangement& a, int D) { return D == 128 ? a.NS128 : a.NS64; }

struct AttnPlan {
  int arr;                     // index into kArrangements
  int WR, WK, NS, threads, wg_per_cu;
  int G, M, RB, nRB, S, chunk;
  int nwork, grid;             // work items, launched workgroups (x8 padded)
  int fused;                   // S > 1: merge in the main kernel's last chunk
  int spread;                  // work order of several sequences (below)
  size_t ws_o_bytes, ws_ml_bytes, ws_sync_bytes, ws_bytes;
  size_t lds_bytes;            // dynamic LDS of the main kernel
  int qshare;                  // key group 0 loads the queries, the others read them from LDS
};

// Dynamic LDS of the main kernel: the rings, then (qshare) the block's
// queries, then the tree tables; the key-group merge reuses it afterwards.
inline size_t attn_lds_bytes(int D, int WR, int WK, int NS, int G, int N, bool qshare) {
  const int RB = kRowsPerWave * WR;
  const size_t stage = 2 * (size_t)kKeyTile * 2 * D;
  const size_t ring = (size_t)WK * NS * stage + (qshare ? (size_t)RB * D * 2 : 0);
  const int words = cdiv(N, 32);
  const int nodes = RB / G + 2;
  const size_t tree = (size_t)nodes * words * 4 + (size_t)N * 4 + 16;
  const size_t waves = (size_t)WR * WK;
  const size_t merge = WK == 1 ? 0 : waves * kRowsPerWave * D * 4 + waves * kRowsPerWave * 8;
  const size_t a = ring + tree;
  return a > merge ? a : merge;
}

// The plan for one arrangement: split count and sizes (grid sized to fill
// every CU with its workgroups-per-CU).
inline AttnPlan attn_plan_arr(int B, int N, int Hq, int Hkv, int D, int Lmax, int arr) {
  const Arrangement& ar = kArrangements[arr];
  AttnPlan p{};
  p.arr = arr;
  p.WR = ar.WR;
  p.WK = ar.WK;
  p.NS = arr_stages(ar, D);
  p.threads = 64 * ar.WR * ar.WK;
  p.wg_per_cu = kWavesPerCU / (ar.WR * ar.WK);
  p.G = Hq / Hkv;
  p.M = N * p.G;
  p.RB = kRowsPerWave * ar.WR;
  p.nRB = cdiv(p.M, p.RB);
  const int tiles = cdiv(Lmax, kKeyTile) + cdiv(N, kKeyTile);
  const long long base = (long long)B * Hkv * p.nRB;
  const long long target = 256LL * p.wg_per_cu;  // every CU full
  const int min_chunk = 2 * ar.WK;               // >= 2 tiles per key group
  long long S = (target + base - 1) / base;
  const long long max_s = tiles / min_chunk > 1 ? tiles / min_chunk : 1;
  if (S > max_s) S = max_s;
  // ragged batches with too few row blocks to fill the GPU: split further so
  // that long sequences spread over several CUs
  if (B > 1 && base < target && S < 4 && max_s >= 4) S = 4;
  if (S < 1 || base > kSyncGroups) S = 1;
  p.chunk = cdiv(tiles, S);
  p.S = cdiv(tiles, p.chunk);
  p.nwork = (int)(base * p.S);
  p.grid = cdiv(p.nwork, kXcds) * kXcds;
  const int DT = D / 16, NTG = p.RB / 16;
  if (p.S > 1) {
    // sync region (counters, then tree flags), chunk partials: O fragments,
    // then (m, l) per row
    p.ws_sync_bytes = kSyncBytes;
    p.ws_o_bytes = (size_t)B * Hkv * p.nRB * p.S * DT * NTG * 64 * 16;
    p.ws_ml_bytes = (size_t)B * Hkv * p.nRB * p.S * p.RB * 8;
  }
  p.ws_bytes = p.ws_sync_bytes + p.ws_o_bytes + p.ws_ml_bytes;
  // The last chunk of a row block merges all of them when that takes at
  // most kFusedMergeBytes of loads per thread (two batches of loads per
  // lane); larger merges go to a second kernel that spreads them over the
  // whole GPU.  1 KB rather than 512 B puts the 4-chunk ragged batch of
  // 16 x 64 nodes (Hq 32, Hkv 4) in the kernel: 1.2% faster than its merge
  // kernel, which had to wait for the slowest sequence.
  p.fused = p.S > 1 && (size_t)p.S * p.RB * D * 4 <= (size_t)kFusedMergeBytes * p.threads;
  // With several key groups every one of them needs the block's queries.
  // When the grid fills every CU, key group 0 loads them and shares them
  // through LDS where that fits: the other groups' copies were 64 KB of
  // requests per workgroup ahead of the first tiles at the Qwen3-8B-shaped
  // 64-node call (2 x 4 waves; 2% faster shared).  On a GPU left mostly
  // idle the copies cost nothing and the LDS hop only adds latency (3%
  // slower for a grid of two workgroups).
  p.qshare = 0;
  p.lds_bytes = p.NS > 0 ? attn_lds_bytes(D, ar.WR, ar.WK, p.NS, p.G, N, false) : kMaxLds + 1;
  if (p.NS > 0 && ar.WK > 1 && ar.WR > 1 && p.nwork >= 256LL * p.wg_per_cu) {
    const size_t with_q = attn_lds_bytes(D, ar.WR, ar.WK, p.NS, p.G, N, true);
    if (with_q * p.wg_per_cu <= kMaxLds) {
      p.qshare = 1;
      p.lds_bytes = with_q;
    }
  }
  // Workgroups go to the XCDs round-robin, and the row blocks of one
  // (sequence, KV head, chunk) read the same keys, so they stay on one XCD
  // (its L2).  With one sequence, XCD x takes a contiguous run of work
  // items.  With several sequences of different lengths that would give
  // each XCD whole sequences and very different work, so each XCD instead
  // takes one KV head and one of L = 8/Hkv lanes of chunks: chunk s of
  // sequence b goes to lane (b + s) % L.  Every XCD then sees every
  // sequence.  This needs Hkv to divide 8 and L to divide S.
  p.spread = B > 1 && kXcds % Hkv == 0 && p.S % (kXcds / Hkv) == 0;
  // Within an XCD workgroups start in index order as slots free up, so a
  // long chunk that starts in a late round sets the kernel's end.  When an
  // XCD's (sequence, chunk) pairs fit the ranking (kMaxRankPairs, tile
  // counts below 2^14), each workgroup ranks them by their tile counts (from
  // kv_len, on the device) and takes the pair whose rank is its position:
  // the longest chunks start first (spread = 2).
  if (p.spread && (long long)B * (p.S / (kXcds / Hkv)) <= kMaxRankPairs && p.chunk < (1 << 14))
    p.spread = 2;
  return p;
}

// The work item (sequence b, KV head g, row block rb, chunk s) of launched
// workgroup `bid`; false for padding workgroups past the work.  constexpr,
// so the kernels and the host checks decode with this same function.  With
// spread = 2 the kernel then replaces the (b, s) pair by the pair of the
// same XCD lane whose length rank is this one's index: a permutation of the
// lane's pairs, so every work item is still covered once.
struct WorkItem {
  int b, g, rb, s;
};
constexpr bool work_item(int grid, int nwork, int S, int nRB, int spread, int B, int Hkv, int bid,
                         WorkItem& it) {
  const int x = bid % kXcds, j = bid / kXcds;
  if (spread) {
    const int L = kXcds / Hkv, per_b = S / L;
    it.g = x % Hkv;
    it.rb = j % nRB;
    const int uu = j / nRB;
    it.b = uu / per_b;
    it.s = ((x / Hkv - it.b) % L + L) % L + L * (uu % per_b);
    return it.b < B;
  }
  int w = x * (grid / kXcds) + j;
  if (w >= nwork) return false;
  it.s = w % S;
  w /= S;
  it.rb = w % nRB;
  w /= nRB;
  it.g = w % Hkv;
  it.b = w / Hkv;
  return it.b < B;
}

inline bool attn_plan_fits(const AttnPlan& p) {
  return p.NS > 0 && p.lds_bytes * p.wg_per_cu <= kMaxLds;
}

// Rough time of an arrangement: matrix work on padded rows, K/V traffic
// from L2 (each row block re-reads the keys), HBM, the split partials
// written and read back, a penalty when the two waves of a SIMD belong
// to one workgroup (its per-tile barriers keep them in phase, so their
// matrix and vector work overlap poorly), and a fixed cost per round of
// workgroups (prologue, first tile's latency, epilogue: a few us each).
inline double attn_plan_cost(const AttnPlan& p, int B, int Hkv, int D, int Lmax, int N) {
  const double keys = (double)Lmax + N;
  double mfma = (double)B * Hkv * p.nRB * p.RB * keys * 4.0 * D / 2.0e15;
  if (p.wg_per_cu == 1 && p.WR > 1) mfma *= 1.3;
  const double kv = (double)B * Hkv * keys * D * 4.0;
  const double l2 = kv * p.nRB / 20.0e12;
  const double hbm = kv / 6.0e12;
  const double partial = (double)p.ws_bytes * 2.0 / 5.0e12;
  const double rounds = (double)cdiv(p.nwork, 256LL * p.wg_per_cu);
  double t = mfma > l2 ? mfma : l2;
  t = t > hbm ? t : hbm;
  return t + partial + rounds * 4.0e-6;
}

inline AttnPlan attn_plan(int B, int N, int Hq, int Hkv, int D, int Lmax) {
  AttnPlan best{};
  double best_cost = 0;
  bool have = false;
  for (int k = 0; k < kNumArrangements; ++k) {
    const AttnPlan p = attn_plan_arr(B, N, Hq, Hkv, D, Lmax, k);
    if (!attn_plan_fits(p)) continue;
    const double c = attn_plan_cost(p, B, Hkv, D, Lmax, N);
    if (!have || c < best_cost) {
      best = p;
      best_cost = c;
      have = true;
    }
  }
  return best;
}

// Acceptance decomposition: a scan kernel runs one workgroup per (node row,
// vocabulary split) and stores one 64-bit key per pair; a second kernel runs
// one workgroup per sequence.  Splits give the scan >= ~2048 workgroups but
// each thread gets at least one full round of kAcceptScanLoads loads.
constexpr int kAcceptMaxSplit = 16;
constexpr int kScanThreads = 256;
constexpr int kScanLoadsPerThread = 8;   // 16-byte loads a thread keeps in flight
// The greedy acceptance scan moves the same bytes per round with twice the
// waves, each keeping half the loads in flight: measured 1-4% faster than
// 256 x 8, while 128 x 16 and 64 x 32 were 5-20% slower.
constexpr int kAcceptScanThreads = 512;
constexpr int kAcceptScanLoads = 4;
static_assert(kAcceptScanThreads * kAcceptScanLoads == kScanThreads * kScanLoadsPerThread,
              "same bytes per round as the other scans");
// The non-greedy acceptance's log-sum-exp scan takes the same shape: 512 x 4
// was 1.6 us faster than 256 x 8 per call at 512 rows of 151936 bf16 logits
// (together with the split rule of sample_plan), the same at 64 rows.
constexpr int kLseScanThreads = 512;
constexpr int kLseScanLoads = 4;
static_assert(kLseScanThreads * kLseScanLoads == kScanThreads * kScanLoadsPerThread,
              "same bytes per round as the other scans");

inline long long accept_split_cap(long long rows) {
  long long ns = (2048 + rows - 1) / rows;
  return ns < 1 ? 1 : (ns > kAcceptMaxSplit ? kAcceptMaxSplit : ns);
}

struct AcceptPlan {
  int nsplit;
  long long chunks_per_split;   // vector chunks (or scalars) per split
  int grid;
  size_t ws_bytes;
};

// Share of a workgroup's load slots that carry data when a row of `chunks`
// vector chunks is cut into ns splits (whole rounds of per_round chunks per
// workgroup; the last round is partly empty).
inline double accept_round_fill(long long chunks, long long ns, long long per_round) {
  const long long c = (chunks + ns - 1) / ns;
  const long long rounds = (c + per_round - 1) / per_round;
  return (double)c / (double)(rounds * per_round);
}

inline AcceptPlan accept_plan(int B, int N, int V, int esize, int vec_elems) {
  AcceptPlan p{};
  const long long rows = (long long)B * N;
  const long long chunks = (V + vec_elems - 1) / vec_elems;
  // at least one full round of loads per thread in every split
  long long ns = accept_split_cap(rows);
  const long long per_round = (long long)kAcceptScanThreads * kAcceptScanLoads;
  const long long by_size = (chunks + per_round - 1) / per_round;
  if (ns > by_size) ns = by_size;
  if (ns < 1) ns = 1;
  // Down to half as many splits, the count whose load slots are best used
  // (ties: more splits): a partly filled last round costs a whole round of
  // latency.  512 rows of 151936 bf16 logits in 4 splits take 2.3 rounds per
  // thread (77% of the slots used), in 2 splits 4.6 (93%), and the
  // acceptance ran 32.6 us in 4 against 31.7 us in 2; 128 rows stay at 10
  // splits (0.93 of one round), where 8 splits (1.16 rounds, 58%) were 5%
  // slower.
  {
    long long best = ns;
    double best_fill = accept_round_fill(chunks, ns, per_round);
    for (long long k = ns - 1; k >= 1 && 2 * k >= ns; --k) {
      const double f = accept_round_fill(chunks, k, per_round);
      if (f > best_fill + 1e-9) {
        best = k;
        best_fill = f;
      }
    }
    ns = best;
  }
  p.chunks_per_split = (chunks + ns - 1) / ns;
  p.nsplit = (int)((chunks + p.chunks_per_split - 1) / p.chunks_per_split);
  p.grid = (int)(rows * p.nsplit);
  p.ws_bytes = (size_t)rows * p.nsplit * 8;
  (void)esize;
  return p;
}

// Workspace bound valid for every dtype and alignment.
inline size_t accept_ws_bytes(int B, int N) {
  const long long rows = (long long)B * N;
  return (size_t)(rows * accept_split_cap(rows) * 8);
}

// Draft top-W (tree drafting's candidates): one workgroup per (draft-depth
// row, vocabulary split) reduces its slice to a running log-sum-exp state
// and its W best (value, token) pairs; a second kernel merges the splits of
// each row.  Splits as in the acceptance scan.
constexpr int kTopwMax = 16;             // largest branching width W
constexpr int kMaxDraftDepth = 64;       // == TV_MAX_DRAFT_DEPTH
constexpr size_t kTopwPartBytes = 8 + 8 * kTopwMax;

struct TopwPlan {
  int nsplit;
  long long chunks_per_split;
  int grid;
  size_t ws_bytes;
};

inline TopwPlan topw_plan(int B, int Nd, int V, int vec_elems) {
  TopwPlan p{};
  const long long rows = (long long)B * Nd;
  const long long chunks = (V + vec_elems - 1) / vec_elems;
  long long ns = accept_split_cap(rows);
  const long long per_round = (long long)kScanThreads * kScanLoadsPerThread;
  const long long by_size = (chunks + per_round - 1) / per_round;
  if (ns > by_size) ns = by_size;
  if (ns < 1) ns = 1;
  p.chunks_per_split = (chunks + ns - 1) / ns;
  p.nsplit = (int)((chunks + p.chunks_per_split - 1) / p.chunks_per_split);
  p.grid = (int)(rows * p.nsplit);
  p.ws_bytes = (size_t)rows * p.nsplit * kTopwPartBytes;
  return p;
}

inline size_t topw_ws_bytes(int B, int Nd) {
  const long long rows = (long long)B * Nd;
  return (size_t)(rows * accept_split_cap(rows)) * kTopwPartBytes;
}

// Non-greedy acceptance: an lse scan over the B*N target rows (splits as
// in the acceptance scan, in vocabulary entries that are multiples of 8),
// then one workgroup per (sequence, race split) that repeats the tests and
// races its vocabulary slice (about 512 workgroups in all, at least 8
// entries per thread, at most kRaceSlice entries so that the slice's token
// mask fits in LDS).
constexpr int kMaxRaceSplit = 64;
constexpr long long kRaceSlice = 131072;
constexpr long long kMaxSampledVocab = kRaceSlice * kMaxRaceSplit;

struct SamplePlan {
  int nsplit, nrace, lse_grid;
  long long eps, rps;  // vocabulary entries per lse / race split
  size_t race_bytes, ws_bytes;
};

inline SamplePlan sample_plan(int B, int N, int V) {
  SamplePlan p{};
  const long long rows = (long long)B * N;
  long long ns = accept_split_cap(rows);
  const long long per_round = (long long)kScanThreads * kScanLoadsPerThread * 8;
  const long long by_size = ((long long)V + per_round - 1) / per_round;
  if (ns > by_size) ns = by_size;
  if (ns < 1) ns = 1;
  {
    // the split count that uses the largest share of its load slots, down
    // to half the workgroup target (as in accept_plan)
    long long best = ns;
    double best_fill = accept_round_fill(V, ns, per_round);
    for (long long k = ns - 1; k >= 1 && 2 * k >= ns; --k) {
      const double f = accept_round_fill(V, k, per_round);
      if (f > best_fill + 1e-9) {
        best = k;
        best_fill = f;
      }
    }
    ns = best;
  }
  p.eps = ((V + ns - 1) / ns + 7) / 8 * 8;
  p.nsplit = (int)((V + p.eps - 1) / p.eps);
  p.lse_grid = (int)(rows * p.nsplit);
  long long nr = (512 + B - 1) / B;
  const long long by_v = ((long long)V + 8 * 256 - 1) / (8 * 256);
  if (nr > by_v) nr = by_v;
  const long long by_mask = ((long long)V + kRaceSlice - 1) / kRaceSlice;
  if (nr < by_mask) nr = by_mask;
  if (nr > kMaxRaceSplit) nr = kMaxRaceSplit;
  if (nr < 1) nr = 1;
  p.rps = ((V + nr - 1) / nr + 7) / 8 * 8;
  p.nrace = (int)((V + p.rps - 1) / p.rps);
  p.race_bytes = ((size_t)B * p.nrace * 16 + 255) / 256 * 256;
  p.ws_bytes = p.race_bytes + (size_t)rows * p.nsplit * 8;
  return p;
}

// LDS of the acceptance of one sequence of N nodes: per node the
// pointer-jumping state (two packed 32-bit words, double-buffered), the
// target argmax (int) and the parent (short).
constexpr size_t accept_lds_bytes(int N) { return (size_t)N * 14 + 16; }

}  // namespace tv
