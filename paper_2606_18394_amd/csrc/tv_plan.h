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
// A workgroup takes RB consecutive rows and one of S contiguous ranges of the
// key tiles (cache tiles first, then tree tiles).
struct AttnPlan {
  int G, M, RB, nRB, S;
  int nwork, grid;             // work items, launched workgroups (x8 padded)
  size_t ws_o_bytes, ws_ml_bytes, ws_bytes;
  size_t lds_bytes;            // dynamic LDS of the main kernel
};

inline size_t attn_lds_bytes(int D, int RB, int G, int N) {
  const size_t vstride = (size_t)D * 2 + 32;
  const size_t staging = (size_t)kWaves * kKeyTile * vstride;
  const int words = cdiv(N, 32);
  const int nodes = RB / G + 2;
  const size_t tree = (size_t)nodes * words * 4 + (size_t)N * 4 + 16;
  const size_t merge = (size_t)kWaves * RB * D * 4 + (size_t)kWaves * RB * 8;
  const size_t a = staging + tree;
  return a > merge ? a : merge;
}

inline AttnPlan attn_plan(int B, int N, int Hq, int Hkv, int D, int Lmax) {
  AttnPlan p{};
  p.G = Hq / Hkv;
  p.M = N * p.G;
  p.RB = p.M <= 32 ? 32 : 64;
  p.nRB = cdiv(p.M, p.RB);
  const int tiles = cdiv(Lmax, kKeyTile) + cdiv(N, kKeyTile);
  const long long base = (long long)B * Hkv * p.nRB;
  const long long target = 2 * 256;          // workgroups wanted in flight
  int S = (int)((target + base - 1) / base);
  const int max_s = tiles / (2 * kWaves) > 1 ? tiles / (2 * kWaves) : 1;
  if (S > max_s) S = max_s;
  if (S < 1) S = 1;
  p.S = S;
  p.nwork = (int)(base * S);
  p.grid = cdiv(p.nwork, kXcds) * kXcds;
  const int DT = D / 16, NT = p.RB / 16;
  if (S > 1) {
    p.ws_o_bytes = (size_t)B * Hkv * p.nRB * S * DT * NT * 64 * 16;
    p.ws_ml_bytes = (size_t)B * Hkv * p.nRB * S * p.RB * 8;
  }
  p.ws_bytes = p.ws_o_bytes + p.ws_ml_bytes;
  p.lds_bytes = attn_lds_bytes(D, p.RB, p.G, N);
  return p;
}

// Acceptance decomposition: each (node row, vocab split) pair is one
// workgroup; the last workgroup of a sequence finishes the sequence.
struct AcceptPlan {
  int nsplit;
  long long chunks_per_split;   // vector chunks (or scalars) per split
  int grid;
  size_t part_bytes, ticket_bytes, ws_bytes;
};

inline AcceptPlan accept_plan(int B, int N, int V, int esize, int vec_elems) {
  AcceptPlan p{};
  const long long rows = (long long)B * N;
  const long long chunks = (V + vec_elems - 1) / vec_elems;
  const long long row_bytes = (long long)V * esize;
  // aim for >= 2048 workgroups but keep >= 32 KB of logits per workgroup
  long long ns = (2048 + rows - 1) / rows;
  long long cap = row_bytes / 32768;
  if (cap < 1) cap = 1;
  if (ns > cap) ns = cap;
  if (ns > chunks) ns = chunks;
  if (ns < 1) ns = 1;
  p.nsplit = (int)ns;
  p.chunks_per_split = (chunks + ns - 1) / ns;
  p.grid = (int)(rows * ns);
  p.part_bytes = (size_t)rows * ns * 8;
  p.ticket_bytes = ((size_t)B * 4 + 255) / 256 * 256;
  p.ws_bytes = p.ticket_bytes + p.part_bytes;
  return p;
}

// Workspace bound valid for every dtype and alignment: nsplit never exceeds
// ceil(2048 / rows).
inline size_t accept_ws_bytes(int B, int N) {
  const long long rows = (long long)B * N;
  long long ns = (2048 + rows - 1) / rows;
  if (ns < 1) ns = 1;
  return ((size_t)B * 4 + 255) / 256 * 256 + (size_t)(rows * ns * 8);
}

}  // namespace tv
