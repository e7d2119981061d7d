// The cache side of a verification step on CDNA4 (gfx950): the accepted
// path's keys and values (root first) are appended to the sequence's cache
// at positions kv_len .. kv_len + accept_len - 1 and kv_len grows by
// accept_len (App. E: the accepted path is committed; paged caches).
//
// One workgroup per sequence.  The rows of the path are copied with 16-byte
// loads and stores spread over all threads; the sequence's kv_len is read
// by every thread before the workgroup barrier and rewritten by one thread
// after it, so a sequence is handled entirely by its own workgroup.  A
// sequence whose acceptance failed (accept_len < 1 or > Dmax), whose path
// names a node outside [0, N) or whose commit would pass the capacity is
// left unchanged.
//
// Tree-tail layout (no separate tree K/V: node i sits at cache row
// kv_len + i): the commit moves rows within the cache, row kv_len + j taking
// row kv_len + path[j].  A root-to-node path has path[j] >= j, so taking the
// rows in increasing j never reads a row after it was overwritten; the copy
// runs in rounds in that order, each round reading all its rows before the
// workgroup barrier and writing them after it.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tv {

struct CommitArgs {
  const uint4* kt;
  const uint4* vt;
  const int32_t* path;
  const int32_t* accept_len;
  uint4* kc;
  uint4* vc;
  int32_t* kv_len;
  const int32_t* block_table;  // paged: [B, max_blocks], else NULL
  int shift, max_blocks, num_blocks;
  int N, cpr, cap, Dmax;  // cpr: 16-byte chunks per row (Hkv * D * 2 / 16)
};

// Row of cache position pos of sequence b (paged: through the block table,
// block numbers clamped into the pool).
__device__ __forceinline__ size_t cache_row(const CommitArgs& a, int b, int pos) {
  if (a.block_table) {
    int blk = a.block_table[(size_t)b * a.max_blocks + (pos >> a.shift)];
    blk = blk < 0 ? 0 : (blk >= a.num_blocks ? a.num_blocks - 1 : blk);
    return ((size_t)blk << a.shift) + (pos & ((1 << a.shift) - 1));
  }
  return (size_t)b * a.cap + pos;
}

constexpr int kTailBatch = 4;  // 16-byte pieces per thread per round of a tree-tail commit

__global__ __launch_bounds__(256) void commit_path(CommitArgs a) {
  const int b = blockIdx.x, tid = threadIdx.x;
  const bool tail = a.kt == nullptr;
  const int kl = a.kv_len[b];
  const int n = a.accept_len[b];
  const int32_t* path = a.path + (size_t)b * a.Dmax;
  // a tree tail needs its N rows inside the capacity
  int bad = n < 1 || n > a.Dmax || kl < 0 || kl > a.cap - (tail ? a.N : n);
  if (!bad)
    for (int j = tid; j < n; j += 256) bad |= path[j] < 0 || path[j] >= a.N;
  if (__syncthreads_or(bad)) return;
  const int per = n * a.cpr;  // chunks of K (or of V)
  if (!tail) {
    for (int c = tid; c < 2 * per; c += 256) {
      const bool isv = c >= per;
      const int r = isv ? c - per : c;
      const int j = r / a.cpr, q = r % a.cpr;
      const size_t src = ((size_t)b * a.N + path[j]) * a.cpr + q;
      const size_t dst = cache_row(a, b, kl + j) * a.cpr + q;
      if (isv) a.vc[dst] = a.vt[src];
      else a.kc[dst] = a.kt[src];
    }
  } else {
    // piece c: row j = c / (2 cpr), then K or V, then the 16-byte piece
    const int rowp = 2 * a.cpr;
    for (int c0 = 0; c0 < 2 * per; c0 += kTailBatch * 256) {
      uint4 v[kTailBatch];
      size_t dst[kTailBatch];
      bool isv[kTailBatch];
#pragma unroll
      for (int u = 0; u < kTailBatch; ++u) {
        const int c = c0 + u * 256 + tid;
        if (c < 2 * per) {
          const int j = c / rowp, r = c % rowp;
          isv[u] = r >= a.cpr;
          const int q = isv[u] ? r - a.cpr : r;
          const size_t src = cache_row(a, b, kl + path[j]) * a.cpr + q;
          dst[u] = cache_row(a, b, kl + j) * a.cpr + q;
          v[u] = isv[u] ? a.vc[src] : a.kc[src];
        }
      }
      __syncthreads();  // the round's reads are done before any of its writes
#pragma unroll
      for (int u = 0; u < kTailBatch; ++u) {
        const int c = c0 + u * 256 + tid;
        if (c < 2 * per) {
          if (isv[u]) a.vc[dst[u]] = v[u];
          else a.kc[dst[u]] = v[u];
        }
      }
      __syncthreads();
    }
  }
  __syncthreads();  // every thread has read kv_len
  if (tid == 0) a.kv_len[b] = kl + n;
}

hipError_t launch_commit(const void* kt, const void* vt, const int32_t* path,
                         const int32_t* accept_len, void* kc, void* vc, int32_t* kv_len,
                         const int32_t* block_table, int shift, int max_blocks, int num_blocks,
                         int B, int N, int Hkv, int D, int cap, int Dmax, hipStream_t st) {
  CommitArgs a;
  a.kt = (const uint4*)kt;
  a.vt = (const uint4*)vt;
  a.path = path;
  a.accept_len = accept_len;
  a.kc = (uint4*)kc;
  a.vc = (uint4*)vc;
  a.kv_len = kv_len;
  a.block_table = block_table;
  a.shift = shift;
  a.max_blocks = max_blocks;
  a.num_blocks = num_blocks;
  a.N = N;
  a.cpr = Hkv * D * 2 / 16;
  a.cap = cap;
  a.Dmax = Dmax;
  hipLaunchKernelGGL(commit_path, dim3(B), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace tv
