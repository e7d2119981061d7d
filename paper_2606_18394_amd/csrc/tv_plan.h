// Host-side launch planning shared by the entry points and the kernels'
// launchers.  Pure C++ (no HIP): the plans depend only on host-known sizes.
#pragma once
#include <stddef.h>
#include <stdint.h>

namespace tv {

constexpr int kWaves = 4;          // waves per attention workgroup
constexpr int kKeyTile = 32;       // keys one wave consumes per step
constexpr int kXcds = 8;           // MI355X accelerator complex dies
constexpr int kMaxNodes = 2048;    // == TV_MAX_NODES

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Attention work decomposition.  Rows of one (sequence, KV head) pair are the
// N*G (node, query-head-in-group) pairs, row r = node * G + head_in_group.
// A workgroup takes one block of consecutive rows (64 in keys mode, 256 in
// rows mode) and one fixed-size chunk of the key tiles (cache tiles first,
// then tree tiles).
constexpr int kKeysModeRB = 64;
constexpr int kRowsModeRB = 256;

// LDS ring depth (stages of one 32-key K tile + V tile)
constexpr int ring_stages(int D, bool rows_mode) {
  return rows_mode ? 4 : (D == 128 ? 2 : 4);
}

struct AttnPlan {
  bool rows_mode;
  int G, M, RB, nRB, S, chunk;
  int nwork, grid;             // work items, launched workgroups (x8 padded)
  size_t ws_o_bytes, ws_ml_bytes, ws_bytes;
  size_t lds_bytes;            // dynamic LDS of the main kernel
};

inline size_t attn_lds_bytes(int D, bool rows_mode, int G, int N) {
  const int RB = rows_mode ? kRowsModeRB : kKeysModeRB;
  const size_t stage = 2 * (size_t)kKeyTile * 2 * D;
  const size_t ring = (rows_mode ? 1 : kWaves) * (size_t)ring_stages(D, rows_mode) * stage;
  const int words = cdiv(N, 32);
  const int nodes = RB / G + 2;
  const size_t tree = (size_t)nodes * words * 4 + (size_t)N * 4 + 16;
  const size_t merge = rows_mode ? 0 : (size_t)kWaves * RB * D * 4 + (size_t)kWaves * RB * 8;
  const size_t a = ring + tree;
  return a > merge ? a : merge;
}

inline AttnPlan attn_plan(int B, int N, int Hq, int Hkv, int D, int Lmax) {
  AttnPlan p{};
  p.G = Hq / Hkv;
  p.M = N * p.G;
  p.rows_mode = p.M >= 2 * kRowsModeRB;
  p.RB = p.rows_mode ? kRowsModeRB : kKeysModeRB;
  p.nRB = cdiv(p.M, p.RB);
  const int tiles = cdiv(Lmax, kKeyTile) + cdiv(N, kKeyTile);
  const long long base = (long long)B * Hkv * p.nRB;
  const long long target = 256;                 // one workgroup per CU
  const int min_chunk = p.rows_mode ? 4 : 2 * kWaves;
  long long S = (target + base - 1) / base;
  const long long max_s = tiles / min_chunk > 1 ? tiles / min_chunk : 1;
  if (S > max_s) S = max_s;
  if (S < 1) S = 1;
  p.chunk = cdiv(tiles, S);
  p.S = cdiv(tiles, p.chunk);
  p.nwork = (int)(base * p.S);
  p.grid = cdiv(p.nwork, kXcds) * kXcds;
  const int DT = D / 16, NTG = p.RB / 16;
  if (p.S > 1) {
    p.ws_o_bytes = (size_t)B * Hkv * p.nRB * p.S * DT * NTG * 64 * 16;
    p.ws_ml_bytes = (size_t)B * Hkv * p.nRB * p.S * p.RB * 8;
  }
  p.ws_bytes = p.ws_o_bytes + p.ws_ml_bytes;
  p.lds_bytes = attn_lds_bytes(D, p.rows_mode, p.G, N);
  return p;
}

// Acceptance decomposition: a scan kernel runs one workgroup per (node row,
// vocabulary split) and writes one 64-bit key per pair; a finish kernel runs
// one workgroup per sequence.  Splits give the scan >= ~2048 workgroups but
// each thread gets at least one full round of kScanLoadsPerThread loads.
constexpr int kAcceptMaxSplit = 16;
constexpr int kScanThreads = 256;
constexpr int kScanLoadsPerThread = 8;   // 16-byte loads a thread keeps in flight

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

inline AcceptPlan accept_plan(int B, int N, int V, int esize, int vec_elems) {
  AcceptPlan p{};
  const long long rows = (long long)B * N;
  const long long chunks = (V + vec_elems - 1) / vec_elems;
  // at least one full round of loads per thread in every split
  long long ns = accept_split_cap(rows);
  const long long per_round = (long long)kScanThreads * kScanLoadsPerThread;
  const long long by_size = (chunks + per_round - 1) / per_round;
  if (ns > by_size) ns = by_size;
  if (ns < 1) ns = 1;
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

}  // namespace tv
