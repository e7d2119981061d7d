// Greedy tree acceptance for CDNA4 (gfx950).
//
// The target's greedy prediction at node i is the first index of the
// maximum of its logits; draft node i is accepted when its token equals the
// prediction at its parent and the parent is accepted; the result is the
// deepest accepted root-to-node path (Sec. 2.4 greedy rule; App. E).
//
// Two kernels, no global atomics:
//   scan    one workgroup per (node row, vocabulary split).  256 threads
//           stream their slice with 16-byte loads, kScanLoadsPerThread of
//           them in flight per thread, and keep a running first maximum;
//           the workgroup reduces it with wave64 shuffles on the 64-bit key
//             key = order-preserving(value) << 32 | (0xFFFFFFFF - index)
//           whose maximum is the largest value at its lowest index (-0.0 is
//           folded into +0.0 first, so equal values compare equal), and
//           stores the key in the workspace.
//   finish  one workgroup per sequence: merges the split keys into the
//           per-node argmax, validates the tree, computes acceptance for all
//           nodes at once by pointer jumping over the parent links
//           (O(log depth) rounds), picks the deepest accepted node (lowest
//           index on ties) and writes the path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tv_plan.h"

namespace tv {

struct AcceptArgs {
  const void* logits;
  const int32_t* draft;
  const int32_t* parent;
  int32_t* accept_len;
  int32_t* path;
  int32_t* tgt_out;
  unsigned long long* part;
  int B, N, V, Dmax, nsplit;
  long long cps;  // chunks per split
};

__device__ __forceinline__ unsigned long long make_key(float v, unsigned int idx) {
  unsigned int u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;                       // -0.0 -> +0.0
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);     // monotone in value
  return ((unsigned long long)u << 32) | (unsigned long long)(0xFFFFFFFFu - idx);
}

__device__ __forceinline__ unsigned long long umax64(unsigned long long x, unsigned long long y) {
  return x > y ? x : y;
}

__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long k) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned int lo = __shfl_xor((unsigned int)k, o);
    const unsigned int hi = __shfl_xor((unsigned int)(k >> 32), o);
    k = umax64(k, ((unsigned long long)hi << 32) | lo);
  }
  return k;
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

template <bool F32, bool VEC>
__global__ __launch_bounds__(kScanThreads) void accept_scan(AcceptArgs a) {
  constexpr int E = VEC ? (F32 ? 4 : 8) : 1;  // elements per chunk
  constexpr int L = kScanLoadsPerThread;
  const int tid = threadIdx.x;
  const int row = blockIdx.x / a.nsplit;       // b * N + i
  const int split = blockIdx.x % a.nsplit;
  const long long nchunks = ((long long)a.V + E - 1) / E;
  const long long c0 = (long long)split * a.cps;
  const long long c1 = c0 + a.cps < nchunks ? c0 + a.cps : nchunks;

  Best best{0.f, 0u, false};
  if (VEC) {
    const uint4* base = reinterpret_cast<const uint4*>(
        (const char*)a.logits + (size_t)row * a.V * (F32 ? 4 : 2));
    // rounds of L loads per thread, all issued before any is used
    for (long long c = c0 + tid; c < c1; c += (long long)L * kScanThreads) {
      uint4 w[L];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kScanThreads;
        if (cu < c1) w[u] = base[cu];
      }
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kScanThreads;
        if (cu < c1) see_chunk<F32>(best, w[u], (unsigned int)(cu * E));
      }
    }
  } else {
    for (long long c = c0 + tid; c < c1; c += kScanThreads) {
      float x;
      if (F32) {
        x = reinterpret_cast<const float*>(a.logits)[(size_t)row * a.V + c];
      } else {
        const unsigned short h =
            reinterpret_cast<const unsigned short*>(a.logits)[(size_t)row * a.V + c];
        x = __uint_as_float((unsigned int)h << 16);
      }
      best.see(x, (unsigned int)c);
    }
  }

  __shared__ unsigned long long red[kScanThreads / 64];
  unsigned long long key = best.any ? make_key(best.v, best.i) : 0ull;
  key = wave_max_u64(key);
  if ((tid & 63) == 0) red[tid >> 6] = key;
  __syncthreads();
  if (tid == 0) {
    key = red[0];
#pragma unroll
    for (int k = 1; k < kScanThreads / 64; ++k) key = umax64(key, red[k]);
    a.part[(size_t)row * a.nsplit + split] = key;
  }
}

__global__ __launch_bounds__(256) void accept_finish(AcceptArgs a) {
  __shared__ short par[kMaxNodes];
  __shared__ int tgt[kMaxNodes];
  __shared__ unsigned long long rowkey[kMaxNodes];
  __shared__ unsigned char ok[2][kMaxNodes];
  __shared__ short jmp[2][kMaxNodes];
  __shared__ short dep[2][kMaxNodes];
  __shared__ unsigned int best_key;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const int N = a.N;
  // parents and drafts of this thread's nodes: loads issued first
  int pv[kMaxNodes / 256], dv[kMaxNodes / 256];
#pragma unroll
  for (int k = 0; k < kMaxNodes / 256; ++k) {
    const int i = tid + 256 * k;
    pv[k] = i < N ? a.parent[(size_t)b * N + i] : 0;
    dv[k] = i < N ? a.draft[(size_t)b * N + i] : 0;
  }
  // the split keys of all rows, merged with LDS max; loads go out in
  // batches of kFinishLoads so their latencies overlap
  constexpr int kFinishLoads = 8;
  for (int i = tid; i < N; i += 256) rowkey[i] = 0ull;
  __syncthreads();
  const size_t kbase = (size_t)b * N * a.nsplit;
  const int nkeys = N * a.nsplit;
  for (int idx0 = 0; idx0 < nkeys; idx0 += 256 * kFinishLoads) {
    unsigned long long kv[kFinishLoads];
#pragma unroll
    for (int u = 0; u < kFinishLoads; ++u) {
      const int idx = idx0 + 256 * u + tid;
      kv[u] = idx < nkeys ? a.part[kbase + idx] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < kFinishLoads; ++u) {
      const int idx = idx0 + 256 * u + tid;
      if (idx < nkeys) atomicMax(&rowkey[idx / a.nsplit], kv[u]);
    }
  }
  int bad = 0;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kMaxNodes / 256; ++k) {
    const int i = tid + 256 * k;
    if (i >= N) break;
    const unsigned long long key = rowkey[i];
    const int t = (int)(0xFFFFFFFFu - (unsigned int)key);
    tgt[i] = t;
    if (a.tgt_out) a.tgt_out[(size_t)b * N + i] = t;
    const int p = pv[k];
    const int badi = (i == 0) ? (p != -1) : (p < 0 || p >= i);
    bad |= badi;
    par[i] = (short)(badi ? 0 : p);
  }
  if (tid == 0) best_key = 0u;
  bad = __syncthreads_or(bad);
  if (!bad) {
#pragma unroll
    for (int k = 0; k < kMaxNodes / 256; ++k) {
      const int i = tid + 256 * k;
      if (i >= N) break;
      if (i == 0) {
        ok[0][0] = 1;
        jmp[0][0] = 0;
        dep[0][0] = 0;
      } else {
        ok[0][i] = dv[k] == tgt[par[i]];
        jmp[0][i] = par[i];
        dep[0][i] = 1;
      }
    }
    __syncthreads();
    // pointer jumping: afterwards jmp = root, dep = depth and ok = every
    // node on the root path matches the prediction at its parent
    int cur = 0, more;
    do {
      const int nxt = cur ^ 1;
      more = 0;
      for (int i = tid; i < N; i += 256) {
        const int j = jmp[cur][i];
        ok[nxt][i] = ok[cur][i] & ok[cur][j];
        dep[nxt][i] = dep[cur][i] + dep[cur][j];
        jmp[nxt][i] = jmp[cur][j];
        more |= jmp[nxt][i] != 0;
      }
      cur = nxt;
    } while (__syncthreads_or(more));
    unsigned int mk = 0u;
    for (int i = tid; i < N; i += 256)
      if (ok[cur][i]) {
        const unsigned int k = ((unsigned int)dep[cur][i] << 16) | (0xFFFFu - (unsigned int)i);
        mk = mk > k ? mk : k;
      }
    atomicMax(&best_key, mk);  // LDS atomic, one per thread
    __syncthreads();
  }
  const unsigned int bk = best_key;
  const int depth = (int)(bk >> 16);
  const int len = bad || depth + 1 > a.Dmax ? -1 : depth + 1;
  int32_t* pth = a.path + (size_t)b * a.Dmax;
  for (int k = tid; k < a.Dmax; k += 256)
    if (k >= len) pth[k] = -1;  // len == -1 clears the whole row
  if (tid == 0) {
    if (len > 0) {
      int u = (int)(0xFFFFu - (bk & 0xFFFFu));
      for (int k = depth; k >= 0; --k) {
        pth[k] = u;
        u = par[u];
      }
    }
    a.accept_len[b] = len;
  }
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
  const dim3 g(p.grid), t(kScanThreads);
  if (f32) {
    if (vec) hipLaunchKernelGGL((accept_scan<true, true>), g, t, 0, st, a);
    else hipLaunchKernelGGL((accept_scan<true, false>), g, t, 0, st, a);
  } else {
    if (vec) hipLaunchKernelGGL((accept_scan<false, true>), g, t, 0, st, a);
    else hipLaunchKernelGGL((accept_scan<false, false>), g, t, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(accept_finish, dim3(B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace tv
