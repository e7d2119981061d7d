// Greedy tree acceptance for CDNA4 (gfx950).
//
// The target's greedy prediction at node i is the first index of the
// maximum of its logits; draft node i is accepted when its token equals the
// prediction at its parent and the parent is accepted; the result is the
// deepest accepted root-to-node path (Sec. 2.4 greedy rule; App. E).
//
// Scan: one workgroup per (node row, vocabulary split).  512 threads stream
// the slice with 16-byte loads, kAcceptScanLoads of them in flight per
// thread, and keep a running first maximum; the workgroup reduces it with
// wave64 shuffles on the 64-bit key
//     key = order-preserving(value) << 32 | (0xFFFFFFFF - index)
// whose maximum is the largest value at its lowest index (-0.0 is folded
// into +0.0 first, so equal values compare equal).
//
// Acceptance of a sequence (one workgroup): validate the parent array,
// compute acceptance for all nodes at once by pointer jumping over the
// parent links (O(log depth) rounds), pick the deepest accepted node (lowest
// index on ties) and write the path.
//
// Two kernels: the scan stores one key per (row, split); one wave (trees of
// up to 128 nodes) or one workgroup per sequence merges its rows' keys in
// registers and runs the acceptance.  A single kernel in which the split
// that completes a row merges it and the row that completes a sequence runs
// its acceptance (device-scope key and prediction stores, per-row and
// per-sequence arrival counters) was parity-green and slower on every
// workload: 16.2 / 20.8 / 62.1 / 39.9 us against 9.4 / 13.4 / 56.1 / 38.1 us
// for 64 / 128 / 16 x 64 / 512 nodes over 151936 bf16 logits.  Its chain of
// dependent device-scope round trips outlasts the kernel boundary it saves.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tv_plan.h"
#include "tv_stream.h"
#include "tv_walk.h"

namespace tv {

struct AcceptArgs {
  const void* logits;
  const int32_t* draft;
  const int32_t* parent;
  int32_t* accept_len;
  int32_t* path;
  int32_t* tgt_out;
  unsigned long long* part;  // split keys [rows, nsplit]
  int B, N, V, Dmax, nsplit;
  long long cps;  // chunks per split
};

__device__ __forceinline__ unsigned long long make_key(float v, unsigned int idx) {
  unsigned int u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;                       // -0.0 -> +0.0
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);     // monotone in value
  return ((unsigned long long)u << 32) | (unsigned long long)(0xFFFFFFFFu - idx);
}

__device__ __forceinline__ int key_index(unsigned long long key) {
  return (int)(0xFFFFFFFFu - (unsigned int)key);
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long x, unsigned long long y) {
  return x > y ? x : y;
}

template <int CTRL>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long k) {
  return ((unsigned long long)dpp_u32<CTRL>((unsigned int)(k >> 32)) << 32) | dpp_u32<CTRL>((unsigned int)k);
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ unsigned long long dpp_bcast_u64(unsigned long long k) {
  return ((unsigned long long)dpp_bcast_u32<CTRL, ROWMASK>((unsigned int)(k >> 32)) << 32) |
         dpp_bcast_u32<CTRL, ROWMASK>((unsigned int)k);
}
// wave_max_u32's DPP steps on a 64-bit key; wave-uniform result
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long k) {
  k = umax64(k, dpp_u64<0xB1>(k));
  k = umax64(k, dpp_u64<0x4E>(k));
  k = umax64(k, dpp_u64<0x141>(k));
  k = umax64(k, dpp_u64<0x140>(k));
  k = umax64(k, dpp_bcast_u64<0x142, 0xA>(k));
  k = umax64(k, dpp_bcast_u64<0x143, 0xC>(k));
  // readlane returns int: widen through unsigned int, not by sign extension
  const unsigned int hi = (unsigned int)__builtin_amdgcn_readlane((unsigned int)(k >> 32), 63);
  const unsigned int lo = (unsigned int)__builtin_amdgcn_readlane((unsigned int)k, 63);
  return ((unsigned long long)hi << 32) | lo;
}

// Running first maximum over a thread's elements, visited in increasing
// index order: only a strictly larger value replaces the current best.
struct Best {
  float v;
  unsigned int i;
  bool any;
  __device__ __forceinline__ void see(float x, unsigned int idx) {
    if (!any || x > v) {
      v = x;
      i = idx;
      any = true;
    }
  }
};

template <bool F32>
__device__ __forceinline__ void see_chunk(Best& best, const uint4& w, unsigned int i0) {
  const unsigned int ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (F32) {
      best.see(__uint_as_float(ws[k]), i0 + k);
    } else {
      best.see(__uint_as_float(ws[k] << 16), i0 + 2 * k);
      best.see(__uint_as_float(ws[k] & 0xFFFF0000u), i0 + 2 * k + 1);
    }
  }
}

// The key of one (row, split) slice, returned to every thread.
template <bool F32, bool VEC>
__device__ __forceinline__ unsigned long long scan_slice(const AcceptArgs& a, int row, int split) {
  constexpr int E = VEC ? (F32 ? 4 : 8) : 1;  // elements per chunk
  constexpr int L = kAcceptScanLoads;
  const int tid = threadIdx.x;
  const long long nchunks = ((long long)a.V + E - 1) / E;
  const long long c0 = (long long)split * a.cps;
  const long long c1 = c0 + a.cps < nchunks ? c0 + a.cps : nchunks;

  Best best{0.f, 0u, false};
  if (VEC) {
    const uint4* base = reinterpret_cast<const uint4*>(
        (const char*)a.logits + (size_t)row * a.V * (F32 ? 4 : 2));
    // rounds of L loads per thread, all issued before any is used
    for (long long c = c0 + tid; c < c1; c += (long long)L * kAcceptScanThreads) {
      uint4 w[L];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kAcceptScanThreads;
        if (cu < c1) w[u] = load_stream(base + cu);
      }
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kAcceptScanThreads;
        if (cu < c1) see_chunk<F32>(best, w[u], (unsigned int)(cu * E));
      }
    }
  } else {
    for (long long c = c0 + tid; c < c1; c += kAcceptScanThreads) {
      float x;
      if (F32) {
        x = load_stream(reinterpret_cast<const float*>(a.logits) + (size_t)row * a.V + c);
      } else {
        const unsigned short h =
            load_stream(reinterpret_cast<const unsigned short*>(a.logits) + (size_t)row * a.V + c);
        x = __uint_as_float((unsigned int)h << 16);
      }
      best.see(x, (unsigned int)c);
    }
  }

  __shared__ unsigned long long red[kAcceptScanThreads / 64];
  unsigned long long key = best.any ? make_key(best.v, best.i) : 0ull;
  key = wave_max_u64(key);
  if ((tid & 63) == 0) red[tid >> 6] = key;
  __syncthreads();
  key = red[0];
#pragma unroll
  for (int k = 1; k < kAcceptScanThreads / 64; ++k) key = umax64(key, red[k]);
  return key;
}

// Threads of the one-workgroup acceptance of trees over 64 nodes (512
// measured faster than 256 or 1024 at 128 and 512 nodes).
constexpr int kFinishThreads = 512;
static_assert(kMaxNodes % kFinishThreads == 0, "whole node batches per thread");

// Per-node LDS arrays of one sequence's acceptance (accept_lds_bytes): the
// prediction, the parent, and the pointer-jumping state packed into one
// word per node (double-buffered), so a round reads a node's whole state
// and its jump target's with one access each.
struct SeqLds {
  int* tgt;
  short* par;
  unsigned int *st0, *st1;
};

__device__ __forceinline__ SeqLds seq_lds(unsigned char* base, int N) {
  SeqLds l;
  l.st0 = reinterpret_cast<unsigned int*>(base);
  l.st1 = l.st0 + N;
  l.tgt = reinterpret_cast<int*>(l.st1 + N);
  l.par = reinterpret_cast<short*>(l.tgt + N);
  return l;
}

__device__ __forceinline__ void load_nodes(const AcceptArgs& a, int b, int (&pv)[kMaxNodes / kFinishThreads],
                                           int (&dv)[kMaxNodes / kFinishThreads]) {
#pragma unroll
  for (int k = 0; k < kMaxNodes / kFinishThreads; ++k) {
    const int i = threadIdx.x + kFinishThreads * k;
    pv[k] = i < a.N ? a.parent[(size_t)b * a.N + i] : 0;
    dv[k] = i < a.N ? a.draft[(size_t)b * a.N + i] : 0;
  }
}

// Acceptance of sequence b once l.tgt holds every node's prediction; pv and
// dv hold parent and draft token of nodes tid + kFinishThreads k.  Called by
// all threads of the workgroup.
__device__ __forceinline__ void accept_sequence(const AcceptArgs& a, int b, const SeqLds& l,
                                                const int (&pv)[kMaxNodes / kFinishThreads],
                                                const int (&dv)[kMaxNodes / kFinishThreads]) {
  __shared__ unsigned int best_key;
  const int tid = threadIdx.x;
  const int N = a.N;
  int bad = 0;
#pragma unroll
  for (int k = 0; k < kMaxNodes / kFinishThreads; ++k) {
    const int i = tid + kFinishThreads * k;
    if (i >= N) break;
    const int p = pv[k];
    const int badi = (i == 0) ? (p != -1) : (p < 0 || p >= i);
    bad |= badi;
    l.par[i] = (short)(badi ? 0 : p);
  }
  if (tid == 0) best_key = 0u;
  bad = __syncthreads_or(bad);
  if (!bad) {
#pragma unroll
    for (int k = 0; k < kMaxNodes / kFinishThreads; ++k) {
      const int i = tid + kFinishThreads * k;
      if (i >= N) break;
      // the root (par = -1) jumps to itself
      const int p = i == 0 ? 0 : l.par[i];
      l.st0[i] = pack_state((unsigned int)p, i == 0 ? 0u : 1u, i == 0 || dv[k] == l.tgt[p]);
    }
    __syncthreads();
    // pointer jumping: afterwards every node jumps to the root with its
    // depth, and ok = every node on its root path matches the prediction at
    // its parent.  Jumps double each round, so ceil(log2(kMaxNodes)) = 11
    // rounds reach the root from any node; the round cap only bounds the loop.
    int cur = 0, more, rounds = 0;
    do {
      const unsigned int* sc = cur ? l.st1 : l.st0;
      unsigned int* sn = cur ? l.st0 : l.st1;
      more = 0;
      for (int i = tid; i < N; i += kFinishThreads) {
        const unsigned int w = jump_state(sc, i);
        sn[i] = w;
        more |= (w & kJmpMask) != 0;
      }
      cur ^= 1;
    } while (__syncthreads_or(more) && ++rounds < 16);
    const unsigned int* sc = cur ? l.st1 : l.st0;
    unsigned int mk = 0u;
    for (int i = tid; i < N; i += kFinishThreads) {
      const unsigned int k = deepest_key(sc[i], i);
      mk = mk > k ? mk : k;
    }
    // the wave's maximum first: same-address LDS atomics serialise, and one
    // per thread took 2 us of the 512-node acceptance
    mk = wave_max_u32(mk);
    if ((tid & 63) == 0) atomicMax(&best_key, mk);
    __syncthreads();
  }
  const unsigned int bk = best_key;
  const int depth = (int)(bk >> 16);
  const int len = bad || depth + 1 > a.Dmax ? -1 : depth + 1;
  int32_t* pth = a.path + (size_t)b * a.Dmax;
  for (int k = tid; k < a.Dmax; k += kFinishThreads)
    if (k >= len) pth[k] = -1;  // len == -1 clears the whole row
  if (tid == 0) {
    if (len > 0) {
      int u = (int)(0xFFFFu - (bk & 0xFFFFu));
      for (int k = depth; k >= 0; --k) {
        pth[k] = u;
        u = l.par[u];
      }
    }
    a.accept_len[b] = len;
  }
}

// First kernel: the key of every (row, split).
template <bool F32, bool VEC>
__global__ __launch_bounds__(kAcceptScanThreads) void accept_scan(AcceptArgs a) {
  const int row = blockIdx.x / a.nsplit;
  const int split = blockIdx.x % a.nsplit;
  const unsigned long long key = scan_slice<F32, VEC>(a, row, split);
  if (threadIdx.x == 0) a.part[(size_t)row * a.nsplit + split] = key;
}

// Second kernel: one workgroup per sequence; thread t takes rows t,
// t + kFinishThreads, ...: it requests every split key of its row at once
// (only the plan's splits: the split count is the same for every thread,
// so the loads past it are skipped by a uniform branch; at 512 nodes in 2
// splits that took the acceptance from 31.7 to 31.1 us, against loads of
// all 16 slots at clamped indices), keeps the max in registers, and the
// acceptance runs on the merged predictions.  The parents and tokens are requested first, so all of the
// kernel's global loads are in flight together.
__global__ __launch_bounds__(kFinishThreads) void accept_finish(AcceptArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int N = a.N;
  constexpr int kRows = kMaxNodes / kFinishThreads;
  int pv[kRows], dv[kRows];
  load_nodes(a, b, pv, dv);
  const SeqLds l = seq_lds(lds, N);
#pragma unroll
  for (int k = 0; k < kRows; ++k) {
    const int i = tid + kFinishThreads * k;
    if (i < N) {
      const unsigned long long* kp = a.part + ((size_t)b * N + i) * a.nsplit;
      unsigned long long kv[kAcceptMaxSplit];
#pragma unroll
      for (int s = 0; s < kAcceptMaxSplit; ++s) kv[s] = s < a.nsplit ? kp[s] : 0ull;
      unsigned long long key = 0ull;
#pragma unroll
      for (int s = 0; s < kAcceptMaxSplit; ++s) key = umax64(key, kv[s]);
      const int t = key_index(key);
      l.tgt[i] = t;
      if (a.tgt_out) a.tgt_out[(size_t)b * N + i] = t;
    }
  }
  __syncthreads();
  accept_sequence(a, b, l, pv, dv);
}

// Split keys a node's merge requests: the plans give trees of more than
// 32 * NPL nodes at most min(16, 64 / NPL) splits (the acceptance plan
// aims at about 2048 (row, split) pairs and caps splits at 16).
template <int NPL>
constexpr int wave_finish_loads() {
  return 64 / NPL < kAcceptMaxSplit ? 64 / NPL : kAcceptMaxSplit;
}

// The value of node j (held by lane j % 64 in slot j / 64).  Every lane
// takes part in every exchange (an inactive source lane would read as
// zero), so the slot is selected after the shuffles.
template <int NPL>
__device__ __forceinline__ int lane_fetch(const int (&v)[NPL], int j) {
  const int src = j & 63, slot = j >> 6;
  int r = __shfl(v[0], src);
#pragma unroll
  for (int q = 1; q < NPL; ++q) {
    const int t = __shfl(v[q], src);
    r = slot == q ? t : r;
  }
  return r;
}

// Loads issued as inline assembly, so that the compiler neither waits for
// them where it would (before work that does not use them) nor moves their
// uses; completion is awaited with explicit vmcnt waits (loads return in
// issue order), after which `loaded` ties each value to the wait.
__device__ __forceinline__ int ld_i32(const int32_t* p) {
  int v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
__device__ __forceinline__ unsigned long long ld_u64(const unsigned long long* p) {
  unsigned long long v;
  asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}
template <class T>
__device__ __forceinline__ void loaded(T& v) {
  asm volatile("" : "+v"(v));
}
// s_waitcnt vmcnt(n) with the other counters left alone (gfx9 encoding)
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Second kernel for trees of at most 64 * NPL nodes (NPL = 1 or 2): one
// wave per sequence, lane l holding nodes l, l + 64, ..., l + 64 (NPL - 1),
// so everything runs on lane exchanges: no LDS and no workgroup barrier.
// The tree's shape needs only the parents, so while the split keys are in
// flight, pointer jumping over the parent links gives every node its
// ancestor-or-self set as a bitmask of 64 * NPL bits (its depth is the
// set's size minus one).  Once the keys are in, one ballot per slot gives
// the nodes whose token equals the prediction at their parent (the root
// always passes); a node is accepted iff its set holds no node outside
// that ballot, the deepest accepted node (lowest index on ties) ends the
// path, and every node of its set writes its own path entry.  Same results
// as accept_finish.
template <int NPL>
__global__ __launch_bounds__(64) void accept_finish_wave(AcceptArgs a) {
  constexpr int NW = 2 * NPL;  // 32-bit words of a node set
  const int b = blockIdx.x, lane = threadIdx.x;
  const int N = a.N;
  int p[NPL], y[NPL], tgt[NPL], jmp[NPL];
  int anc[NW][NPL];  // word w of the ancestor-or-self set of node lane + 64 q
  bool node[NPL];
  int badi = 0;
  // Requests, oldest first: the parents, each node's split keys (indices
  // past the last split repeat it, which leaves the max unchanged), the
  // draft tokens.  Padding lanes read node N - 1's; nothing of theirs is
  // used.  The parents are awaited before the shape is built, the rest only
  // after it, so the keys arrive while the lanes exchange parent links.
  constexpr int kLoads = wave_finish_loads<NPL>();
  unsigned long long kv[NPL][kLoads];
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    const int i = lane + 64 * q;
    node[q] = i < N;
    p[q] = ld_i32(a.parent + (size_t)b * N + (node[q] ? i : N - 1));
  }
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    const int i = lane + 64 * q;
    const unsigned long long* kp = a.part + ((size_t)b * N + (node[q] ? i : N - 1)) * a.nsplit;
#pragma unroll
    for (int k = 0; k < kLoads; ++k) kv[q][k] = ld_u64(kp + min(k, a.nsplit - 1));
  }
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    const int i = lane + 64 * q;
    y[q] = ld_i32(a.draft + (size_t)b * N + (node[q] ? i : N - 1));
  }
  wait_vm<NPL * kLoads + NPL>();
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    loaded(p[q]);
    if (!node[q]) p[q] = 0;
  }
  // the shape: valid parents, then pointer jumping on (jump target,
  // ancestor set); the root and padding jump to node 0, whose set is {0}
  int more = 0;
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    const int i = lane + 64 * q;
    const int bq = node[q] && ((i == 0) ? (p[q] != -1) : (p[q] < 0 || p[q] >= i));
    badi |= bq;
    jmp[q] = node[q] && i > 0 && !bq ? p[q] : 0;
    more |= jmp[q] != 0;
#pragma unroll
    for (int w = 0; w < NW; ++w)
      anc[w][q] = !node[q] ? 0 : (int)((w == (i >> 5) ? 1u << (i & 31) : 0u) | (w == 0 ? 1u : 0u));
  }
  const bool bad = __any(badi);
  if (!bad) {
    // every exchange of a round reads the values of the round before;
    // ceil(log2(64 NPL)) rounds reach the root from any node
    for (int r = 0; r < 12 && __any(more); ++r) {
      int aj[NW][NPL], jj[NPL];
#pragma unroll
      for (int q = 0; q < NPL; ++q) {
        jj[q] = lane_fetch<NPL>(jmp, jmp[q]);
#pragma unroll
        for (int w = 0; w < NW; ++w) aj[w][q] = lane_fetch<NPL>(anc[w], jmp[q]);
      }
      more = 0;
#pragma unroll
      for (int q = 0; q < NPL; ++q) {
        jmp[q] = jj[q];
        more |= jmp[q] != 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) anc[w][q] |= aj[w][q];
      }
    }
  }
  // the predictions: the max of each node's split keys
  wait_vm<0>();
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    loaded(y[q]);
#pragma unroll
    for (int k = 0; k < kLoads; ++k) loaded(kv[q][k]);
  }
#pragma unroll
  for (int q = 0; q < NPL; ++q) {
    const int i = lane + 64 * q;
    unsigned long long key = 0ull;
#pragma unroll
    for (int k = 0; k < kLoads; ++k) key = umax64(key, kv[q][k]);
    tgt[q] = key_index(node[q] ? key : 0ull);
    if (node[q] && a.tgt_out) a.tgt_out[(size_t)b * N + i] = tgt[q];
  }
  int len = -1, depth = 0, dep[NPL];
  unsigned int avw[NW];  // the winner's ancestor set
  if (!bad) {
    // nodes that pass: word w of the mask holds nodes 32 w .. 32 w + 31
    unsigned int okw[NW];
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
      const int i = lane + 64 * q;
      const int tp = lane_fetch<NPL>(tgt, node[q] && i > 0 ? p[q] : 0);
      const bool pass = node[q] && (i == 0 || y[q] == tp);
      const unsigned long long m = __ballot(pass);
      okw[2 * q] = (unsigned int)m;
      okw[2 * q + 1] = (unsigned int)(m >> 32);
    }
    unsigned int k = 0u;
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
      const int i = lane + 64 * q;
      unsigned int fail = 0u;
      int cnt = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        fail |= (unsigned int)anc[w][q] & ~okw[w];
        cnt += __popc((unsigned int)anc[w][q]);
      }
      dep[q] = cnt - 1;
      const unsigned int kq =
          node[q] && fail == 0u ? ((unsigned int)dep[q] << 16) | (0xFFFFu - (unsigned int)i) : 0u;
      k = kq > k ? kq : k;
    }
    k = wave_max_u32(k);
    depth = (int)(k >> 16);
    const int v = (int)(0xFFFFu - (k & 0xFFFFu));
    len = depth + 1 > a.Dmax ? -1 : depth + 1;
#pragma unroll
    for (int w = 0; w < NW; ++w) avw[w] = (unsigned int)lane_fetch<NPL>(anc[w], v);
  }
  int32_t* pth = a.path + (size_t)b * a.Dmax;
  for (int k = lane; k < a.Dmax; k += 64)
    if (k >= len) pth[k] = -1;
  if (len > 0) {
    // the winner's root path: each of its nodes writes the entry at its depth
#pragma unroll
    for (int q = 0; q < NPL; ++q) {
      const int i = lane + 64 * q;
      unsigned int on = 0u;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        if (w == (i >> 5)) on = (avw[w] >> (i & 31)) & 1u;
      if (node[q] && on) pth[dep[q]] = i;
    }
  }
  if (lane == 0) a.accept_len[b] = len;
}

hipError_t launch_accept(const void* logits, int f32, const int32_t* draft, const int32_t* parent,
                         int B, int N, int V, int Dmax, int32_t* accept_len, int32_t* path,
                         int32_t* tgt_out, void* ws, hipStream_t st) {
  const int esize = f32 ? 4 : 2;
  const int velems = 16 / esize;
  const bool vec = ((uintptr_t)logits % 16 == 0) && ((size_t)V * esize % 16 == 0);
  const AcceptPlan p = accept_plan(B, N, V, esize, vec ? velems : 1);
  AcceptArgs a;
  a.logits = logits;
  a.draft = draft;
  a.parent = parent;
  a.accept_len = accept_len;
  a.path = path;
  a.tgt_out = tgt_out;
  a.part = (unsigned long long*)ws;
  a.B = B;
  a.N = N;
  a.V = V;
  a.Dmax = Dmax;
  a.nsplit = p.nsplit;
  a.cps = p.chunks_per_split;
  const dim3 g(p.grid), t(kAcceptScanThreads);
  if (f32) {
    if (vec) hipLaunchKernelGGL((accept_scan<true, true>), g, t, 0, st, a);
    else hipLaunchKernelGGL((accept_scan<true, false>), g, t, 0, st, a);
  } else {
    if (vec) hipLaunchKernelGGL((accept_scan<false, true>), g, t, 0, st, a);
    else hipLaunchKernelGGL((accept_scan<false, false>), g, t, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One wave per sequence up to 128 nodes (the plans' split counts fit its
  // loads, checked here), else a workgroup of kFinishThreads.  At two nodes
  // per lane the wave takes 13.3 us against 17.1 us for the workgroup
  // (long_ctx, 128 nodes); at eight per lane its lane exchanges (eight per
  // value and round) made it 55.8 us against 37.8 us (big_tree_32b).
  if (N <= 64 && p.nsplit <= wave_finish_loads<1>())
    hipLaunchKernelGGL(accept_finish_wave<1>, dim3(B), dim3(64), 0, st, a);
  else if (N <= 128 && p.nsplit <= wave_finish_loads<2>())
    hipLaunchKernelGGL(accept_finish_wave<2>, dim3(B), dim3(64), 0, st, a);
  else
    hipLaunchKernelGGL(accept_finish, dim3(B), dim3(kFinishThreads), accept_lds_bytes(N), st, a);
  return hipGetLastError();
}

}  // namespace tv
