// Budgeted tree drafting for CDNA4 (gfx950): the step that produces the
// trees the verification kernels consume (Sec. 2.4, parallel tree drafting;
// Alg. 1; App. E).
//
// topw: candidate children per draft depth.  One draft-head pass gives a
//   logit row per draft depth; its W largest entries (equal values: lower
//   token id) and their log-probabilities (logit minus the row's
//   log-sum-exp) are the children offered to every node one depth above.
//   Scan: one workgroup per (row, vocabulary split) streams its slice with
//   16-byte loads, keeps a running (max, sum of exponentials) per thread,
//   updated once per batch of loads, and a sorted top-W list in registers;
//   the workgroup merges the lists by W rounds of (value, lower index)
//   argmax.  Finish: one wave per row merges the splits.
//
// build: best-first expansion under a node budget, one wave per sequence.
//   Node i is owned by lane i % 64 (slot i / 64), which keeps the score
//   keys of its open nodes in registers and caches its best one; a pop is a
//   wave maximum of those keys (an order-preserving unsigned image of the
//   fp32 score) with ties settled by the lower node index, the owner
//   rescans its slots in registers, and the up to W children go to W
//   consecutive lanes.  The loop only logs the popped nodes; parents,
//   tokens, depths and scores are rebuilt from that log at the end.  Scores
//   are fp32 sums parent + log-probability, the comparisons that decide the
//   tree.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv_plan.h"
#include "tv_stream.h"
#include "tv_walk.h"

namespace tv {

// ---------------------------------------------------------------- topw

struct TopwArgs {
  const void* logits;
  int32_t* tok;
  float* logp;
  unsigned char* part;  // per (row, split): m, s, then kTopwMax (value, index)
  int rows, V, W, nsplit;
  long long cps;        // chunks per split
};

struct TopwPart {
  float m, s;
  float v[kTopwMax];
  int i[kTopwMax];
};

// Sorted list of the K best (value, index) pairs seen, decreasing, K a
// compile-time length >= W (a list cut at a runtime W would be indexed
// dynamically and live in scratch memory).  Insertion is a branch-free
// bubble pass.  Within a thread, elements arrive in increasing index order,
// so an equal value never displaces an earlier entry (strict comparison).
template <int K>
struct TopList {
  float v[K];
  int i[K];
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      v[k] = -INFINITY;
      i[k] = 0x7FFFFFFF;
    }
  }
  __device__ __forceinline__ float thr() const { return v[K - 1]; }
  __device__ __forceinline__ void insert(float x, int idx) {
    float cv = x;
    int ci = idx;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const bool sw = cv > v[k];
      const float nv = sw ? cv : v[k];
      const int ni = sw ? ci : i[k];
      cv = sw ? v[k] : cv;
      ci = sw ? i[k] : ci;
      v[k] = nv;
      i[k] = ni;
    }
  }
  // drop the head (it was taken by the merge)
  __device__ __forceinline__ void pop() {
#pragma unroll
    for (int k = 0; k < K - 1; ++k) {
      v[k] = v[k + 1];
      i[k] = i[k + 1];
    }
    v[K - 1] = -INFINITY;
    i[K - 1] = 0x7FFFFFFF;
  }
};

__device__ __forceinline__ bool better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

// Wave-wide best (value, lower index); every lane receives the result.
// Within each row of 16 lanes: DPP exchanges with lane ^ 1 and lane ^ 2
// (quad permutes), then mirrored lanes of each half-row and of the row,
// after which all 16 lanes hold the row's best; the four rows are then read
// out as scalars.  (Cross-lane shuffles would go through the LDS crossbar,
// one round trip per step.)
template <int CTRL>
__device__ __forceinline__ int dpp(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ void dpp_best_step(float& v, int& i) {
  const float ov = __int_as_float(dpp<CTRL>(__float_as_int(v)));
  const int oi = dpp<CTRL>(i);
  if (better(ov, oi, v, i)) {
    v = ov;
    i = oi;
  }
}
__device__ __forceinline__ void wave_best(float& v, int& i) {
  dpp_best_step<0xB1>(v, i);   // quad_perm(1,0,3,2): lane ^ 1
  dpp_best_step<0x4E>(v, i);   // quad_perm(2,3,0,1): lane ^ 2
  dpp_best_step<0x141>(v, i);  // row_half_mirror: quads of each half-row
  dpp_best_step<0x140>(v, i);  // row_mirror: the two halves of the row
  float gv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  int gi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const float rv = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), r));
    const int ri = __builtin_amdgcn_readlane(i, r);
    if (better(rv, ri, gv, gi)) {
      gv = rv;
      gi = ri;
    }
  }
  v = gv;
  i = gi;
}

// Order-preserving map of a score to a nonzero key: a larger score gives a
// larger key, so one unsigned maximum compares scores.  (-0.0 would sort
// below +0.0; no score takes that value, since the root's is +0.0 and a
// sum that cancels to zero rounds to +0.0.)  Key 0 marks "no open node".
__device__ __forceinline__ unsigned score_key(float s) {
  const unsigned u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_score(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Wave-wide minimum of an unsigned value (the maximum, wave_max_u32, is in
// tv_walk.h), returned as a wave-uniform value: DPP steps inside each row of
// 16 lanes, then the four rows' values read out as scalars (it runs only on
// ties, off the hot loops).
__device__ __forceinline__ unsigned wave_min_u32(unsigned x) {
  x = min(x, dpp_u32<0xB1>(x));
  x = min(x, dpp_u32<0x4E>(x));
  x = min(x, dpp_u32<0x141>(x));
  x = min(x, dpp_u32<0x140>(x));
  const unsigned r0 = __builtin_amdgcn_readlane(x, 0), r1 = __builtin_amdgcn_readlane(x, 16);
  const unsigned r2 = __builtin_amdgcn_readlane(x, 32), r3 = __builtin_amdgcn_readlane(x, 48);
  return min(min(r0, r1), min(r2, r3));
}

// (m, s) with s = sum exp(x - m): merge of two such states
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __expf(m - mn) + s2 * __expf(m2 - mn);
  m = mn;
}
template <int CTRL>
__device__ __forceinline__ void lse_dpp_step(float& m, float& s) {
  lse_merge(m, s, __int_as_float(dpp<CTRL>(__float_as_int(m))), __int_as_float(dpp<CTRL>(__float_as_int(s))));
}
// Wave-wide merge of (m, s): DPP pair merges inside each row of 16 lanes
// (a merge of two states is symmetric, so both lanes of a pair hold the
// same result), then the four rows' states merged as scalars.
__device__ __forceinline__ void wave_lse(float& m, float& s) {
  lse_dpp_step<0xB1>(m, s);
  lse_dpp_step<0x4E>(m, s);
  lse_dpp_step<0x141>(m, s);
  lse_dpp_step<0x140>(m, s);
  float gm = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), 0));
  float gs = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 0));
#pragma unroll
  for (int r = 16; r < 64; r += 16)
    lse_merge(gm, gs, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), r)),
              __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), r)));
  m = gm;
  s = gs;
}

// Key of a candidate value for the wave maximum: -0.0 counts as +0.0, as
// the float comparison does; an empty entry (-inf at index 0x7FFFFFFF,
// logits being finite) has key 0.
__device__ __forceinline__ unsigned cand_key(float v, int i) {
  return i == 0x7FFFFFFF ? 0u : score_key(v + 0.f);
}
// The lane holding the best (value, lower index) entry among the lanes'
// heads: a wave maximum of the keys; the lanes holding it are a ballot, and
// with several (equal values) the lowest index wins.  -1 if all are empty.
__device__ __forceinline__ int best_head_lane(float v, int i) {
  const unsigned k = cand_key(v, i);
  const unsigned g = wave_max_u32(k);
  if (g == 0u) return -1;
  const unsigned long long hold = __ballot(k == g);
  if (__popcll(hold) == 1) return __ffsll((unsigned long long)hold) - 1;
  const unsigned bi = wave_min_u32(k == g ? (unsigned)i : 0xFFFFFFFFu);
  return __ffsll((unsigned long long)__ballot(k == g && (unsigned)i == bi)) - 1;
}

// Slices of one load round (ONE) rank their candidates directly: every
// element >= tau is appended to an LDS list, and each listed candidate's
// rank is the number of listed candidates better than it; ranks below W are
// the slice's top-W.  More than kTopwCand candidates (values tied at tau)
// fall back to the per-thread lists and W rounds of workgroup argmax.
constexpr int kTopwCand = kScanThreads;

template <bool F32, bool VEC, int K, bool ONE>
__global__ __launch_bounds__(kScanThreads) void topw_scan(TopwArgs a) {
  constexpr int E = VEC ? (F32 ? 4 : 8) : 1;  // elements per chunk
  constexpr int L = kScanLoadsPerThread;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ int s_ncand;
  __shared__ float s_cv[kTopwCand];
  __shared__ int s_ci[kTopwCand];
  if (ONE && tid == 0) s_ncand = 0;  // read after the first round's barrier
  int ncand = 0;
  const int row = blockIdx.x / a.nsplit;
  const int split = blockIdx.x % a.nsplit;
  const long long nchunks = ((long long)a.V + E - 1) / E;
  const long long c0 = (long long)split * a.cps;
  const long long c1 = c0 + a.cps < nchunks ? c0 + a.cps : nchunks;
  const int W = a.W;

  TopList<K> top;
  top.init();
  float m = -INFINITY, s = 0.f;
  // tau: a lower bound on the slice's W-th largest value, known after the
  // first round; only elements >= tau reach the (divergent) list insertion
  float tau = -INFINITY;
  const char* rowp = (const char*)a.logits + (size_t)row * a.V * (F32 ? 4 : 2);
  // rounds are uniform across the workgroup (the first ends at a barrier)
  for (long long cb = c0; cb < c1; cb += (long long)L * kScanThreads) {
    const long long c = cb + tid;
    // all L loads are issued first (past the end: the last chunk again),
    // then decoded with the padding replaced by -inf bit patterns, so the
    // loads are in flight together
    constexpr unsigned int kNegInf = F32 ? 0xFF800000u : 0xFF80FF80u;
    uint4 raw[L];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const long long cu = c + (long long)u * kScanThreads;
      const long long cl = cu < c1 ? cu : c1 - 1;
      if (VEC) {
        raw[u] = load_stream(reinterpret_cast<const uint4*>(rowp) + cl);
      } else if (F32) {
        raw[u].x = load_stream(reinterpret_cast<const unsigned int*>(rowp) + cl);
      } else {
        raw[u].x = (unsigned int)load_stream(reinterpret_cast<const unsigned short*>(rowp) + cl) << 16;
      }
    }
    float x[L][E];
#pragma unroll
    for (int u = 0; u < L; ++u) {
      const bool in = c + (long long)u * kScanThreads < c1;
      const unsigned int ws[4] = {in ? raw[u].x : kNegInf, in ? raw[u].y : kNegInf,
                                  in ? raw[u].z : kNegInf, in ? raw[u].w : kNegInf};
      if (VEC) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (F32) {
            x[u][k] = __uint_as_float(ws[k]);
          } else {
            x[u][2 * k] = __uint_as_float(ws[k] << 16);
            x[u][2 * k + 1] = __uint_as_float(ws[k] & 0xFFFF0000u);
          }
        }
      } else {
        x[u][0] = __uint_as_float(in ? raw[u].x : 0xFF800000u);
      }
    }
    float bmu[L];  // maximum of each load
    float bm = -INFINITY;
#pragma unroll
    for (int u = 0; u < L; ++u) {
      bmu[u] = x[u][0];
#pragma unroll
      for (int e = 1; e < E; ++e) bmu[u] = fmaxf(bmu[u], x[u][e]);
      bm = fmaxf(bm, bmu[u]);
    }
    if (bm != -INFINITY) {  // a thread past the slice end has only padding
      const float mn = fmaxf(m, bm);
      float bs = 0.f;
#pragma unroll
      for (int u = 0; u < L; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) bs += __expf(x[u][e] - mn);  // exp(-inf) = 0 for padding
      s = (m == -INFINITY ? 0.f : s * __expf(m - mn)) + bs;
      m = mn;
    }
    if (cb == c0) {
      // Each wave's q-th largest thread maximum, q = ceil(W / waves): every
      // wave holds q elements at least that large, so at least W elements
      // of the slice are >= the smallest of these.
      constexpr int kWaves = kScanThreads / 64;
      __shared__ float s_tau[kWaves];
      const int q = (W + kWaves - 1) / kWaves;
      // q rounds of a key maximum; one lane holding it drops out each round
      unsigned kv = bm == -INFINITY ? 0u : score_key(bm + 0.f), gk = 0u;
      for (int r = 0; r < q; ++r) {
        gk = wave_max_u32(kv);
        if (gk == 0u) break;  // fewer than q threads with data
        if (lane == __ffsll((unsigned long long)__ballot(kv == gk)) - 1) kv = 0u;
      }
      const float kth = gk == 0u ? -INFINITY : key_score(gk);
      if (lane == 0) s_tau[wave] = kth;
      __syncthreads();
      tau = s_tau[0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) tau = fminf(tau, s_tau[w]);
    }
    if (ONE) {
      // the slice's top-W are all >= tau: list them (not the padding)
      if (bm >= tau) {
#pragma unroll
        for (int u = 0; u < L; ++u) {
          const long long cu = c + (long long)u * kScanThreads;
          if (cu < c1 && bmu[u] >= tau) {
#pragma unroll
            for (int e = 0; e < E; ++e)
              if (x[u][e] >= tau) {
                const int slot = atomicAdd(&s_ncand, 1);
                if (slot < kTopwCand) {
                  s_cv[slot] = x[u][e];
                  s_ci[slot] = (int)(cu * E + e);
                }
              }
          }
        }
      }
      __syncthreads();
      ncand = s_ncand;
    }
    // padding (-inf) never passes; equal values keep the earlier index
    if ((!ONE || ncand > kTopwCand) && bm >= tau && bm > top.thr()) {
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kScanThreads;
#pragma unroll
        for (int e = 0; e < E; ++e)
          if (x[u][e] >= tau && x[u][e] > top.thr()) top.insert(x[u][e], (int)(cu * E + e));
      }
    }
  }

  // workgroup: (m, s) by shuffles and LDS, the top-W by W rounds of argmax
  __shared__ float red_m[kScanThreads / 64], red_s[kScanThreads / 64];
  __shared__ float win_v[kScanThreads / 64];
  __shared__ int win_i[kScanThreads / 64];
  wave_lse(m, s);
  if (lane == 0) {
    red_m[wave] = m;
    red_s[wave] = s;
  }
  TopwPart* out = reinterpret_cast<TopwPart*>(a.part + ((size_t)row * a.nsplit + split) * kTopwPartBytes);
  if (ONE && ncand <= kTopwCand) {
    if (tid < ncand) {
      const float v = s_cv[tid];
      const int i = s_ci[tid];
      int rank = 0;
      for (int j = 0; j < ncand; ++j) rank += better(s_cv[j], s_ci[j], v, i) ? 1 : 0;
      if (rank < W) {
        out->v[rank] = v;
        out->i[rank] = i;
      }
    } else if (tid < W) {  // a slice with fewer than W elements
      out->v[tid] = -INFINITY;
      out->i[tid] = 0x7FFFFFFF;
    }
    __syncthreads();  // the waves' (m, s)
  } else {
    for (int k = 0; k < W; ++k) {
      float bv = top.v[0];
      int bi = top.i[0];
      wave_best(bv, bi);
      if (lane == 0) {
        win_v[wave] = bv;
        win_i[wave] = bi;
      }
      __syncthreads();
      float gv = win_v[0];
      int gi = win_i[0];
#pragma unroll
      for (int w = 1; w < kScanThreads / 64; ++w)
        if (better(win_v[w], win_i[w], gv, gi)) {
          gv = win_v[w];
          gi = win_i[w];
        }
      if (top.i[0] == gi && gi != 0x7FFFFFFF) top.pop();  // indices are unique: one owner
      if (tid == 0) {
        out->v[k] = gv;
        out->i[k] = gi;
      }
      __syncthreads();
    }
  }
  if (tid == 0) {
    float gm = red_m[0], gs = red_s[0];
#pragma unroll
    for (int w = 1; w < kScanThreads / 64; ++w) lse_merge(gm, gs, red_m[w], red_s[w]);
    out->m = gm;
    out->s = gs;
  }
}

// One wave per row: lane j < nsplit holds split j's sorted list.  Each of
// the W rounds takes the best head (one key maximum and a ballot) and the
// owning lane drops it.
template <int K>
__global__ __launch_bounds__(64) void topw_finish(TopwArgs a) {
  const int row = blockIdx.x, lane = threadIdx.x;
  const int W = a.W;
  float m = -INFINITY, s = 0.f;
  TopList<K> top;
  top.init();
  if (lane < a.nsplit) {
    const TopwPart* p =
        reinterpret_cast<const TopwPart*>(a.part + ((size_t)row * a.nsplit + lane) * kTopwPartBytes);
    m = p->m;
    s = p->s;
#pragma unroll
    for (int k = 0; k < K; ++k)
      if (k < W) {
        top.v[k] = p->v[k];
        top.i[k] = p->i[k];
      }
  }
  wave_lse(m, s);
  const float lse = m + logf(s);
  for (int k = 0; k < W; ++k) {
    const int owner = best_head_lane(top.v[0], top.i[0]);
    const float bv = owner < 0 ? -INFINITY : __int_as_float(__builtin_amdgcn_readlane(__float_as_int(top.v[0]), owner < 0 ? 0 : owner));
    const int bi = owner < 0 ? 0x7FFFFFFF : __builtin_amdgcn_readlane(top.i[0], owner < 0 ? 0 : owner);
    if (lane == owner) top.pop();
    if (lane == 0) {
      a.tok[(size_t)row * W + k] = bi;
      a.logp[(size_t)row * W + k] = bv - lse;
    }
  }
}

template <int K, bool ONE>
static void launch_topw_scan_k(bool f32, bool vec, dim3 g, dim3 t, hipStream_t st,
                               const TopwArgs& a) {
  if (f32) {
    if (vec) hipLaunchKernelGGL((topw_scan<true, true, K, ONE>), g, t, 0, st, a);
    else hipLaunchKernelGGL((topw_scan<true, false, K, ONE>), g, t, 0, st, a);
  } else {
    if (vec) hipLaunchKernelGGL((topw_scan<false, true, K, ONE>), g, t, 0, st, a);
    else hipLaunchKernelGGL((topw_scan<false, false, K, ONE>), g, t, 0, st, a);
  }
}

template <bool ONE>
static void launch_topw_scan_one(bool f32, bool vec, int K, dim3 g, dim3 t, hipStream_t st,
                                 const TopwArgs& a) {
  if (K == 4) launch_topw_scan_k<4, ONE>(f32, vec, g, t, st, a);
  else if (K == 8) launch_topw_scan_k<8, ONE>(f32, vec, g, t, st, a);
  else launch_topw_scan_k<kTopwMax, ONE>(f32, vec, g, t, st, a);
}

static void launch_topw_scan(bool f32, bool vec, int K, bool one, dim3 g, dim3 t,
                             hipStream_t st, const TopwArgs& a) {
  if (one) launch_topw_scan_one<true>(f32, vec, K, g, t, st, a);
  else launch_topw_scan_one<false>(f32, vec, K, g, t, st, a);
}

hipError_t launch_topw(const void* logits, int f32, int B, int Nd, int V, int W, int32_t* tok,
                       float* logp, void* ws, hipStream_t st) {
  const int esize = f32 ? 4 : 2;
  const bool vec = ((uintptr_t)logits % 16 == 0) && ((size_t)V * esize % 16 == 0);
  const TopwPlan p = topw_plan(B, Nd, V, vec ? 16 / esize : 1);
  TopwArgs a;
  a.logits = logits;
  a.tok = tok;
  a.logp = logp;
  a.part = (unsigned char*)ws;
  a.rows = B * Nd;
  a.V = V;
  a.W = W;
  a.nsplit = p.nsplit;
  a.cps = p.chunks_per_split;
  const dim3 g(p.grid), t(kScanThreads);
  const int K = W <= 4 ? 4 : (W <= 8 ? 8 : 16);
  // one load round per workgroup: every split's slice fits in one
  const bool one = p.chunks_per_split <= (long long)kScanThreads * kScanLoadsPerThread;
  launch_topw_scan(f32 != 0, vec, K, one, g, t, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (K == 4) hipLaunchKernelGGL(topw_finish<4>, dim3(a.rows), dim3(64), 0, st, a);
  else if (K == 8) hipLaunchKernelGGL(topw_finish<8>, dim3(a.rows), dim3(64), 0, st, a);
  else hipLaunchKernelGGL(topw_finish<kTopwMax>, dim3(a.rows), dim3(64), 0, st, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- build

struct BuildArgs {
  const int32_t* tok;
  const float* logp;
  const int32_t* root_tok;
  int32_t* parent;
  int32_t* token;
  int32_t* depth;
  float* score;
  int32_t* n_nodes;
  int Nd, W, budget;
};

// Best-first expansion for budgets of at most 64 S nodes, one wave per
// sequence.  Node i belongs to lane i % 64, slot i / 64.  A lane keeps, per
// slot, the score key of its node while that node is open (0 otherwise)
// and the slot and depth packed as slot << 8 | depth, plus its best open
// node (largest key, lowest slot on equal keys).  A pop:
//  * the wave maximum of the lanes' best keys; the lanes holding it are a
//    ballot, and with several (equal scores) the lowest node index wins;
//  * the owner closes the node and rescans its slots in registers;
//  * the up to W children go to consecutive lanes: child k of a depth-d
//    node gets key(score + logp[d, k]) if depth d + 1 is below Nd, else 0.
// Every pop but the last adds exactly W children, so node c >= 1 is child
// (c - 1) % W of the ((c - 1) / W)-th popped node: the loop only logs the
// popped nodes (index, depth, key) in LDS, and parents, tokens, depths
// and scores are rebuilt from that log at the end, with the same fp32 sum
// the loop's key came from.
template <int S>
__global__ __launch_bounds__(64) void build_tree(BuildArgs a) {
  static_assert(S >= 1 && S <= kMaxNodes / 64, "slots per lane");
  __shared__ float cand_lp[kMaxDraftDepth * kTopwMax];
  __shared__ int cand_tok[kMaxDraftDepth * kTopwMax];
  __shared__ unsigned pop_key[kMaxNodes];
  __shared__ int pop_node[kMaxNodes];  // node index | depth << 16
  const int b = blockIdx.x, lane = threadIdx.x;
  const int Nd = a.Nd, W = a.W, budget = a.budget;
  const size_t cbase = (size_t)b * Nd * W;
  for (int k = lane; k < Nd * W; k += 64) {
    cand_lp[k] = a.logp[cbase + k];
    cand_tok[k] = a.tok[cbase + k];
  }
  __syncthreads();
  unsigned key[S];
  int sd[S];
#pragma unroll
  for (int j = 0; j < S; ++j) {
    key[j] = 0u;
    sd[j] = 0;
  }
  key[0] = lane == 0 ? score_key(0.f) : 0u;  // the root is open (Nd >= 1)
  unsigned bk = key[0];                       // this lane's best open node:
  int bsd = 0;                                // its key and slot << 8 | depth
  int n = 1, np = 0;
  // each pop adds at least one node, so at most budget - 1 pops
  while (n < budget) {
    const unsigned g = wave_max_u32(bk);
    if (g == 0u) break;  // nothing open
    const unsigned long long hold = __ballot(bk == g);
    int owner;
    if (__popcll(hold) == 1) {
      owner = __ffsll((unsigned long long)hold) - 1;
    } else {  // equal scores: the lowest node index
      const unsigned idx = bk == g ? (unsigned)((bsd >> 8) * 64 + lane) : 0xFFFFFFFFu;
      owner = __builtin_amdgcn_readfirstlane((int)(wave_min_u32(idx) & 63u));
    }
    const int osd = __builtin_amdgcn_readlane(bsd, owner);
    const int jv = osd >> 8, d = osd & 0xFF;
    const int nk = min(W, budget - n);
    const int k = (lane - (n & 63)) & 63;  // this lane's child, if k < nk
    const bool child = k < nk;
    const float lp = cand_lp[d * W + (child ? k : 0)];
    // the owner closes the popped node; every lane rescans (the others
    // find their best unchanged)
    const bool own = lane == owner;
#pragma unroll
    for (int j = 0; j < S; ++j)
      if (own && j == jv) key[j] = 0u;
    unsigned m = key[0];
#pragma unroll
    for (int j = 1; j < S; ++j) m = max(m, key[j]);
    bk = m;
#pragma unroll
    for (int j = S - 1; j >= 0; --j)
      if (key[j] == m) bsd = sd[j];
    const int c = n + k;
    // computed on every lane, so that the LDS read above overlaps the rescan
    unsigned ck = score_key(key_score(g) + lp);
    if (!child || d + 1 >= Nd) ck = 0u;
    const int csd = (c >> 6) << 8 | (d + 1);
    const int jc = child ? c >> 6 : -1;
#pragma unroll
    for (int j = 0; j < S; ++j)
      if (j == jc) {
        key[j] = ck;
        sd[j] = csd;
      }
    if (ck > bk) {  // a child has the lane's highest index: strictly better only
      bk = ck;
      bsd = csd;
    }
    if (lane == 0) {
      pop_key[np] = g;
      pop_node[np] = (jv * 64 + owner) | d << 16;
    }
    ++np;
    n += nk;
  }
  __syncthreads();
  const size_t obase = (size_t)b * budget;
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int c = lane + 64 * j;
    if (c < budget) {
      int par = -1, tk = -1, dep = -1;
      float sc = -INFINITY;
      if (c == 0) {
        tk = a.root_tok ? a.root_tok[b] : -1;
        dep = 0;
        sc = 0.f;
      } else if (c < n) {
        const unsigned t = (unsigned)(c - 1);
        const unsigned p = t / (unsigned)W, kk = t - p * (unsigned)W;
        const int pn = pop_node[p];
        const int pd = pn >> 16;
        par = pn & 0xFFFF;
        tk = cand_tok[pd * W + kk];
        dep = pd + 1;
        sc = key_score(pop_key[p]) + cand_lp[pd * W + kk];
      }
      a.parent[obase + c] = par;
      a.token[obase + c] = tk;
      a.depth[obase + c] = dep;
      if (a.score) a.score[obase + c] = sc;
    }
  }
  if (lane == 0) a.n_nodes[b] = n;
}

hipError_t launch_build_tree(const int32_t* tok, const float* logp, const int32_t* root_tok, int B,
                             int Nd, int W, int budget, int32_t* parent, int32_t* token,
                             int32_t* depth, float* score, int32_t* n_nodes, hipStream_t st) {
  BuildArgs a;
  a.tok = tok;
  a.logp = logp;
  a.root_tok = root_tok;
  a.parent = parent;
  a.token = token;
  a.depth = depth;
  a.score = score;
  a.n_nodes = n_nodes;
  a.Nd = Nd;
  a.W = W;
  a.budget = budget;
  // slots per lane: the fewest that hold the budget
  if (budget <= 64)
    hipLaunchKernelGGL(build_tree<1>, dim3(B), dim3(64), 0, st, a);
  else if (budget <= 128)
    hipLaunchKernelGGL(build_tree<2>, dim3(B), dim3(64), 0, st, a);
  else if (budget <= 256)
    hipLaunchKernelGGL(build_tree<4>, dim3(B), dim3(64), 0, st, a);
  else if (budget <= 512)
    hipLaunchKernelGGL(build_tree<8>, dim3(B), dim3(64), 0, st, a);
  else if (budget <= 1024)
    hipLaunchKernelGGL(build_tree<16>, dim3(B), dim3(64), 0, st, a);
  else
    hipLaunchKernelGGL(build_tree<kMaxNodes / 64>, dim3(B), dim3(64), 0, st, a);
  return hipGetLastError();
}

}  // namespace tv
