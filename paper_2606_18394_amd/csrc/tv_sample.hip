// Non-greedy tree acceptance (temperature T > 0) for CDNA4 (gfx950).
//
// The speculative sampling rule (Sec. 2.4) applied to a tree whose
// children are deterministic drafts (top-W, Alg. 1): each child's proposal
// is the point mass at its token, so the children of the current node v are
// tested in index order against the target residual left by the rejected
// ones -- child c (token y) passes when u_c * (1 - S) < e_c, with
// e_c = p_v(y) for a valid token not already rejected at v and 0 otherwise,
// and S the mass of v's earlier children's distinct tokens -- and the first
// child that passes is followed.  This keeps verification lossless
// (Sec. 2.2).  The walk ends at a node none of whose children passes; the
// correction token is drawn there from p_v without its children's tokens
// (from p_v when that leaves no mass), by an exponential race: the winner
// is argmax w(x) / E_x with E_x = -ln U(b, x), U from Philox4x32-10 (Salmon
// et al., SC 2011) on the counter (x / 4, b, 0, 0) and the 64-bit seed as
// key, word x % 4, mapped to (0, 1) by its top 23 bits.
//
// The walk needs no sequential descent: whether child c passes depends only
// on its earlier siblings, so every node's test is taken at once, a node is
// selected when it passes and no earlier sibling does (an LDS atomicMin per
// parent), and the walk is the chain of nodes whose whole root path is
// selected (an AND over root paths by pointer jumping).
//
// Three kernels:
//   lse_scan: one workgroup per (node row, vocabulary split): running
//     (max, sum of exponentials) of x / T per thread, merged across the
//     workgroup.
//   sample_accept: one workgroup per (sequence, vocabulary split).  Each
//     merges the log-sum-exps of its sequence, takes every node's test,
//     finds the walk's last node and races its vocabulary slice for the
//     correction token with that node's child tokens masked by an LDS
//     bitmap, keeping two keys: the residual race and the plain p_v race.
//     Split 0 writes the path.  Every workgroup of a sequence repeats the
//     tests, which costs less than a kernel boundary between them and the
//     race.
//   sample_finish: one wave per sequence merges the race keys.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv_plan.h"
#include "tv_stream.h"
#include "tv_walk.h"

namespace tv {

struct SampleArgs {
  const void* logits;   // [B, N, V] target
  const int32_t* draft;
  const int32_t* parent;
  const float* u;       // [B, N] acceptance uniforms
  int32_t* accept_len;
  int32_t* path;
  int32_t* corr;
  unsigned long long* race;  // [B, nrace, 2] race keys
  float2* lse_part;          // [B*N, nsplit] (max, sum exp) of x / T
  unsigned int seed_lo, seed_hi;
  float invT;
  int B, N, V, Dmax, nsplit, nrace;
  long long eps;  // vocabulary entries per lse split, a multiple of 8
  long long rps;  // vocabulary entries per race split, a multiple of 8, <= kRaceSlice
};

// ------------------------------------------------------------ generator

constexpr unsigned int kPhiloxM0 = 0xD2511F53u, kPhiloxM1 = 0xCD9E8D57u;
constexpr unsigned int kPhiloxW0 = 0x9E3779B9u, kPhiloxW1 = 0xBB67AE85u;

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, unsigned int k0, unsigned int k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const unsigned int hi0 = __umulhi(kPhiloxM0, c.x), lo0 = kPhiloxM0 * c.x;
    const unsigned int hi1 = __umulhi(kPhiloxM1, c.z), lo1 = kPhiloxM1 * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

// top 23 bits -> (k + 1/2) / 2^23, exact in fp32, inside (0, 1)
__device__ __forceinline__ float open_uniform(unsigned int w) {
  return ((float)(w >> 9) + 0.5f) * (1.0f / 8388608.0f);
}

// ------------------------------------------------------------ helpers

__device__ __forceinline__ void lse_merge2(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __expf(m - mn) + s2 * __expf(m2 - mn);
  m = mn;
}

template <int CTRL>
__device__ __forceinline__ void lse_dpp2(float& m, float& s) {
  lse_merge2(m, s, __uint_as_float(dpp_u32<CTRL>(__float_as_uint(m))),
             __uint_as_float(dpp_u32<CTRL>(__float_as_uint(s))));
}

template <bool F32>
__device__ __forceinline__ float load_logit(const void* base, size_t idx) {
  if (F32) return reinterpret_cast<const float*>(base)[idx];
  return __uint_as_float((unsigned int)reinterpret_cast<const unsigned short*>(base)[idx] << 16);
}

// 8 consecutive logits from a 16-byte aligned position (two loads for fp32)
template <bool F32>
__device__ __forceinline__ void load8(const void* base, size_t idx, float (&x)[8]) {
  if (F32) {
    const uint4* p = reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(base) + idx);
    const uint4 a = p[0], b = p[1];
    const unsigned int w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = __uint_as_float(w[k]);
  } else {
    const uint4 a =
        *reinterpret_cast<const uint4*>(reinterpret_cast<const unsigned short*>(base) + idx);
    const unsigned int w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] = __uint_as_float(w[k] << 16);
      x[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
    }
  }
}

__device__ __forceinline__ unsigned long long race_key(float r, unsigned int x) {
  // r >= 0: its bits order like the value; the low word keeps the lowest
  // index on ties and makes every key of a positive weight nonzero
  return ((unsigned long long)__float_as_uint(r) << 32) | (0xFFFFFFFFu - x);
}

// Wave-wide maximum of a 64-bit key on DPP exchanges (four steps inside
// each row of 16 lanes, then the two row broadcasts into lane 63), returned
// as a wave-uniform value.
__device__ __forceinline__ unsigned long long wave_max_key(unsigned long long k) {
  auto step = [](unsigned long long x, unsigned int hi, unsigned int lo) {
    const unsigned long long o = ((unsigned long long)hi << 32) | lo;
    return o > x ? o : x;
  };
  k = step(k, dpp_u32<0xB1>((unsigned int)(k >> 32)), dpp_u32<0xB1>((unsigned int)k));
  k = step(k, dpp_u32<0x4E>((unsigned int)(k >> 32)), dpp_u32<0x4E>((unsigned int)k));
  k = step(k, dpp_u32<0x141>((unsigned int)(k >> 32)), dpp_u32<0x141>((unsigned int)k));
  k = step(k, dpp_u32<0x140>((unsigned int)(k >> 32)), dpp_u32<0x140>((unsigned int)k));
  k = step(k, dpp_bcast_u32<0x142, 0xA>((unsigned int)(k >> 32)), dpp_bcast_u32<0x142, 0xA>((unsigned int)k));
  k = step(k, dpp_bcast_u32<0x143, 0xC>((unsigned int)(k >> 32)), dpp_bcast_u32<0x143, 0xC>((unsigned int)k));
  // readlane returns int: widen through unsigned int, not by sign extension
  const unsigned int hi = (unsigned int)__builtin_amdgcn_readlane((unsigned int)(k >> 32), 63);
  const unsigned int lo = (unsigned int)__builtin_amdgcn_readlane((unsigned int)k, 63);
  return ((unsigned long long)hi << 32) | lo;
}

// ------------------------------------------------------------ lse_scan

// (max, sum exp) of x / T over elements [x0, x1) of a row, into m and s,
// which start at (-inf, 0); x0 and x1 are multiples of 8 (or x1 = V) so that
// vectorised rows read whole 16-byte chunks of either dtype
template <bool F32>
__device__ __forceinline__ void lse_slice(const void* rowp, long long x0, long long x1, bool vec,
                                          float invT, float& m, float& s) {
  constexpr int E = F32 ? 4 : 8;  // elements per 16-byte chunk
  constexpr int L = kLseScanLoads;
  const int tid = threadIdx.x;
  if (vec) {
    // In base-2 units: with c2 = log2(e) / T a weight is exp2(x * c2 - m2)
    // (one fma and one exp2 per logit), m2 the running maximum of x * c2;
    // the batch maximum is taken on the raw logits (c2 > 0 keeps the order).
    // m is returned in the natural units of x / T.
    const float c2 = invT * 1.4426950408889634f;
    float m2 = -INFINITY;
    const long long c0 = x0 / E, c1 = (x1 + E - 1) / E;
    const uint4* base = reinterpret_cast<const uint4*>(rowp);
    for (long long c = c0 + tid; c < c1; c += (long long)L * kLseScanThreads) {
      // all L loads are issued first (past the end: the last chunk again),
      // then decoded with the padding replaced by -inf bit patterns, so the
      // loads are in flight together
      constexpr unsigned int kNegInf = F32 ? 0xFF800000u : 0xFF80FF80u;
      uint4 raw[L];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kLseScanThreads;
        raw[u] = load_stream(base + (cu < c1 ? cu : c1 - 1));
      }
      float x[L][E];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const bool in = c + (long long)u * kLseScanThreads < c1;
        const unsigned int ws[4] = {in ? raw[u].x : kNegInf, in ? raw[u].y : kNegInf,
                                    in ? raw[u].z : kNegInf, in ? raw[u].w : kNegInf};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (F32) {
            x[u][k] = __uint_as_float(ws[k]);
          } else {
            x[u][2 * k] = __uint_as_float(ws[k] << 16);
            x[u][2 * k + 1] = __uint_as_float(ws[k] & 0xFFFF0000u);
          }
        }
      }
      float bm = -INFINITY;
#pragma unroll
      for (int u = 0; u < L; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) bm = fmaxf(bm, x[u][e]);
      if (bm == -INFINITY) continue;
      const float mn = fmaxf(m2, bm * c2);
      float bs = 0.f;
#pragma unroll
      for (int u = 0; u < L; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) bs += __builtin_amdgcn_exp2f(fmaf(x[u][e], c2, -mn));
      s = (m2 == -INFINITY ? 0.f : s * __builtin_amdgcn_exp2f(m2 - mn)) + bs;
      m2 = mn;
    }
    m = m2 == -INFINITY ? -INFINITY : m2 * 0.6931471805599453f;
  } else {
    for (long long c = x0 + tid; c < x1; c += kLseScanThreads) {
      const float x = load_logit<F32>(rowp, (size_t)c) * invT;
      lse_merge2(m, s, x, 1.f);
    }
  }
}

template <bool F32>
__global__ __launch_bounds__(kLseScanThreads) void lse_scan(SampleArgs a, int vec) {
  const int row = blockIdx.x / a.nsplit, split = blockIdx.x % a.nsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const long long x0 = (long long)split * a.eps;
  const long long x1 = x0 + a.eps < a.V ? x0 + a.eps : a.V;
  float m = -INFINITY, s = 0.f;
  const char* rowp = (const char*)a.logits + (size_t)row * a.V * (F32 ? 4 : 2);
  lse_slice<F32>(rowp, x0, x1, vec != 0, a.invT, m, s);
  __shared__ float rm[kLseScanThreads / 64], rs[kLseScanThreads / 64];
  // pair merges inside each row of 16 lanes on DPP exchanges (a merge is
  // symmetric, so both lanes of a pair hold the same state), then the rows
  lse_dpp2<0xB1>(m, s);
  lse_dpp2<0x4E>(m, s);
  lse_dpp2<0x141>(m, s);
  lse_dpp2<0x140>(m, s);
  float wm = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), 0));
  float ws = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), 0));
#pragma unroll
  for (int r = 16; r < 64; r += 16)
    lse_merge2(wm, ws, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(m), r)),
               __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), r)));
  m = wm;
  s = ws;
  if (lane == 0) {
    rm[wave] = m;
    rs[wave] = s;
  }
  __syncthreads();
  if (tid == 0) {
    float gm = rm[0], gs = rs[0];
#pragma unroll
    for (int w = 1; w < kLseScanThreads / 64; ++w) lse_merge2(gm, gs, rm[w], rs[w]);
    a.lse_part[(size_t)row * a.nsplit + split] = make_float2(gm, gs);
  }
}

// ------------------------------------------------------------ sample_accept

constexpr int kSampleThreads = 512;
constexpr int kNodesPerThread = kMaxNodes / kSampleThreads;
static_assert(kMaxNodes % kSampleThreads == 0, "whole node batches per thread");

template <bool F32>
__global__ __launch_bounds__(kSampleThreads) void sample_accept(SampleArgs a, int vec) {
  __shared__ float lse_t[kMaxNodes];
  __shared__ float ef[kMaxNodes];        // effective mass of each node's token at its parent
  __shared__ int tokl[kMaxNodes];
  __shared__ int first_pass[kMaxNodes];  // per parent: lowest passing child
  __shared__ int cnt[kMaxNodes];         // per parent: children, then slots taken
  __shared__ int start[kMaxNodes + 1];   // per parent: first slot of its children
  __shared__ short grp[kMaxNodes], srt[kMaxNodes];  // children by parent: any order, index order
  __shared__ int wsum[kSampleThreads / 64];
  __shared__ short par[kMaxNodes];
  __shared__ unsigned int st0[kMaxNodes], st1[kMaxNodes];  // pointer-jumping state words
  __shared__ unsigned int mask[kRaceSlice / 32];  // child tokens of the last node, this slice
  __shared__ unsigned int best_key;
  __shared__ unsigned long long red[2][kSampleThreads / 64];

  const int b = blockIdx.x / a.nrace, sp = blockIdx.x % a.nrace;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.N, V = a.V;

  // ---- tree, tokens, log-sum-exps
  int bad = 0;
#pragma unroll
  for (int k = 0; k < kNodesPerThread; ++k) {
    const int i = tid + kSampleThreads * k;
    if (i < N) {
      const int p = a.parent[(size_t)b * N + i];
      const int badi = (i == 0) ? (p != -1) : (p < 0 || p >= i);
      bad |= badi;
      par[i] = (short)(badi || i == 0 ? 0 : p);
      tokl[i] = a.draft[(size_t)b * N + i];
      first_pass[i] = 0x7FFFFFFF;
      const size_t row = (size_t)b * N + i;
      float m = -INFINITY, s = 0.f;
      for (int q = 0; q < a.nsplit; ++q) {
        const float2 ps = a.lse_part[row * a.nsplit + q];
        lse_merge2(m, s, ps.x, ps.y);
      }
      lse_t[i] = m + __logf(s);
    }
  }
  if (tid == 0) best_key = 0u;
  bad = __syncthreads_or(bad);

  int len = -1, v = 0, dv = 0;
  if (!bad) {
    // e: p at the parent of each node's token (0 for a token outside [0, V))
    float e[kNodesPerThread];
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      e[k] = 0.f;
      if (i >= 1 && i < N) {
        const int y = tokl[i], u = par[i];
        if (y >= 0 && y < V)
          e[k] = __expf(load_logit<F32>(a.logits, ((size_t)b * N + u) * V + y) * a.invT -
                        lse_t[u]);
      }
    }
    // The children of every node in index order: a counting sort of the
    // non-root nodes by parent (children counted per parent, a scan for
    // the first slot of each parent's group, slots taken in any order, then
    // each node placed by its rank among its siblings, the number of them
    // with a lower index).  Siblings are then contiguous, so a node's
    // earlier siblings are the slots before it in its group.
    for (int i = tid; i < N; i += kSampleThreads) cnt[i] = 0;
    __syncthreads();
    for (int i = 1 + tid; i < N; i += kSampleThreads) atomicAdd(&cnt[par[i]], 1);
    __syncthreads();
    {
      // exclusive scan of cnt[0 .. N): thread t sums entries 4t .. 4t + 3
      constexpr int kPer = kMaxNodes / kSampleThreads;
      int c[kPer], tot = 0;
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int p = kPer * tid + k;
        c[k] = p < N ? cnt[p] : 0;
        tot += c[k];
      }
      int incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
      }
      if (lane == 63) wsum[wave] = incl;
      __syncthreads();
      int off = incl - tot;
      for (int w = 0; w < wave; ++w) off += wsum[w];
#pragma unroll
      for (int k = 0; k < kPer; ++k) {
        const int p = kPer * tid + k;
        if (p < N) start[p] = off;
        off += c[k];
      }
      if (tid == 0) start[N] = N - 1;  // every non-root node has one parent
    }
    for (int i = tid; i < N; i += kSampleThreads) cnt[i] = 0;
    __syncthreads();
    for (int i = 1 + tid; i < N; i += kSampleThreads) {
      const int p = par[i];
      grp[start[p] + atomicAdd(&cnt[p], 1)] = (short)i;
    }
    __syncthreads();
    int rank[kNodesPerThread];
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      rank[k] = 0;
      if (i >= 1 && i < N) {
        const int p = par[i], s0 = start[p], s1 = start[p + 1];
        int r = 0;
        for (int m = s0; m < s1; ++m) r += grp[m] < i;
        srt[s0 + r] = (short)i;
        rank[k] = r;
      }
    }
    __syncthreads();
    // a token repeated among a node's children has no mass left after its
    // first occurrence
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      if (i >= 1 && i < N) {
        const int s0 = start[par[i]], y = tokl[i];
        bool dup = false;
        for (int m = s0; m < s0 + rank[k]; ++m) dup |= tokl[srt[m]] == y;
        ef[i] = dup ? 0.f : e[k];
      }
    }
    __syncthreads();
    // the test against the residual of the earlier siblings (their masses
    // summed in index order), then the lowest passing child of each parent
    unsigned char pass[kNodesPerThread];
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      pass[k] = 0;
      if (i >= 1 && i < N) {
        const int u = par[i], s0 = start[u];
        float S = 0.f;
        for (int m = s0; m < s0 + rank[k]; ++m) S += ef[srt[m]];
        pass[k] = a.u[(size_t)b * N + i] * (1.f - S) < ef[i];
        if (pass[k]) atomicMin(&first_pass[u], i);
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      if (i < N) {
        // the root (par = 0 here) jumps to itself
        st0[i] = pack_state((unsigned int)par[i], i == 0 ? 0u : 1u,
                            i == 0 || (pass[k] && first_pass[par[i]] == i));
      }
    }
    __syncthreads();
    // pointer jumping: afterwards dep = depth and ok = every node of the
    // root path selected; 11 rounds reach the root from any of 2048 nodes
    int cur = 0, more, rounds = 0;
    do {
      const unsigned int* sc = cur ? st1 : st0;
      unsigned int* sn = cur ? st0 : st1;
      more = 0;
      for (int i = tid; i < N; i += kSampleThreads) {
        const unsigned int w = jump_state(sc, i);
        sn[i] = w;
        more |= (w & kJmpMask) != 0;
      }
      cur ^= 1;
    } while (__syncthreads_or(more) && ++rounds < 16);
    const unsigned int* sc = cur ? st1 : st0;
    // the selected nodes form one chain from the root: its deepest node
    // (the wave's maximum first; one LDS atomic per wave)
    unsigned int mk = 0u;
    for (int i = tid; i < N; i += kSampleThreads) {
      const unsigned int k = deepest_key(sc[i], i);
      mk = mk > k ? mk : k;
    }
    mk = wave_max_u32(mk);
    if (lane == 0) atomicMax(&best_key, mk);
    __syncthreads();
    const unsigned int bk = best_key;
    dv = (int)(bk >> 16);
    v = (int)(0xFFFFu - (bk & 0xFFFFu));
    len = dv + 1 > a.Dmax ? -1 : dv + 1;
  }
  if (sp == 0) {
    int32_t* pth = a.path + (size_t)b * a.Dmax;
    for (int k = tid; k < a.Dmax; k += kSampleThreads)
      if (k >= len) pth[k] = -1;
    if (tid == 0) {
      if (len > 0) {
        int w = v;
        for (int k = dv; k >= 0; --k) {
          pth[k] = w;
          w = par[w];
        }
      }
      a.accept_len[b] = len;
    }
  }
  unsigned long long* out = a.race + ((size_t)b * a.nrace + sp) * 2;
  if (len < 0) {  // no correction token; the finish kernel writes -1
    if (tid == 0) out[0] = out[1] = 0ull;
    return;
  }

  // ---- the race over this split's slice of the vocabulary, v's child
  // tokens (all rejected) masked
  const long long x0 = (long long)sp * a.rps;
  const long long x1 = x0 + a.rps < V ? x0 + a.rps : V;
  const int words = (int)((x1 - x0 + 31) / 32);
  for (int k = tid; k < words; k += kSampleThreads) mask[k] = 0u;
  __syncthreads();
  for (int i = 1 + tid; i < N; i += kSampleThreads)
    if (par[i] == v) {
      const long long y = tokl[i];
      if (y >= x0 && y < x1)
        atomicOr(&mask[(y - x0) >> 5], 1u << ((unsigned int)(y - x0) & 31u));
    }
  __syncthreads();
  const float lv = lse_t[v];
  const size_t prow = ((size_t)b * N + v) * V;
  unsigned long long kres = 0ull, kp = 0ull;
  for (long long xg = x0 + 8ll * tid; xg < x1; xg += 8ll * kSampleThreads) {
    float pl[8];
    if (vec && xg + 8 <= x1) {
      load8<F32>(a.logits, prow + xg, pl);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        pl[e] = xg + e < x1 ? load_logit<F32>(a.logits, prow + xg + e) : -INFINITY;
    }
    // 8 entries from an offset that is a multiple of 8 lie in one mask word
    const unsigned int mbits = mask[(xg - x0) >> 5] >> ((unsigned int)(xg - x0) & 31u);
    const uint4 r0 = philox4x32_10(make_uint4((unsigned int)(xg >> 2), (unsigned int)b, 0u, 0u),
                                   a.seed_lo, a.seed_hi);
    const uint4 r1 = philox4x32_10(
        make_uint4((unsigned int)(xg >> 2) + 1u, (unsigned int)b, 0u, 0u), a.seed_lo, a.seed_hi);
    const unsigned int wd[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (xg + e >= x1) break;
      const float p = __expf(pl[e] * a.invT - lv);
      if (p > 0.f) {
        const unsigned long long k = race_key(p / -__logf(open_uniform(wd[e])),
                                              (unsigned int)(xg + e));
        kp = k > kp ? k : kp;
        if (!((mbits >> e) & 1u)) kres = k > kres ? k : kres;
      }
    }
  }
  kres = wave_max_key(kres);
  kp = wave_max_key(kp);
  if (lane == 0) {
    red[0][wave] = kres;
    red[1][wave] = kp;
  }
  __syncthreads();
  if (tid == 0) {
    unsigned long long g0 = red[0][0], g1 = red[1][0];
#pragma unroll
    for (int w = 1; w < kSampleThreads / 64; ++w) {
      g0 = red[0][w] > g0 ? red[0][w] : g0;
      g1 = red[1][w] > g1 ? red[1][w] : g1;
    }
    out[0] = g0;
    out[1] = g1;
  }
}

// ------------------------------------------------------------ finish

__global__ __launch_bounds__(64) void sample_finish(SampleArgs a) {
  const int b = blockIdx.x, lane = threadIdx.x;
  unsigned long long kres = 0ull, kp = 0ull;
  if (lane < a.nrace) {
    const unsigned long long* k = a.race + ((size_t)b * a.nrace + lane) * 2;
    kres = k[0];
    kp = k[1];
  }
  kres = wave_max_key(kres);
  kp = wave_max_key(kp);
  if (lane == 0) {
    const unsigned long long k = kres ? kres : kp;  // no residual mass: race on p
    a.corr[b] = a.accept_len[b] < 0 || k == 0ull ? -1 : (int)(0xFFFFFFFFu - (unsigned int)k);
  }
}

// ------------------------------------------------------------ launch

template <bool F32>
static hipError_t launch_sample_t(const SampleArgs& a, const SamplePlan& p, int vec,
                                  hipStream_t st) {
  hipLaunchKernelGGL((lse_scan<F32>), dim3(p.lse_grid), dim3(kLseScanThreads), 0, st, a, vec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((sample_accept<F32>), dim3(a.B * p.nrace), dim3(kSampleThreads), 0, st, a,
                     vec);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_finish, dim3(a.B), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sample(const void* logits, int f32, const int32_t* draft,
                         const int32_t* parent, const float* u, unsigned long long seed,
                         float temperature, int B, int N, int V, int Dmax, int32_t* accept_len,
                         int32_t* path, int32_t* corr, void* ws, hipStream_t st) {
  const SamplePlan p = sample_plan(B, N, V);
  const int vec = (uintptr_t)logits % 16 == 0 && V % 8 == 0;
  SampleArgs a;
  a.logits = logits;
  a.draft = draft;
  a.parent = parent;
  a.u = u;
  a.accept_len = accept_len;
  a.path = path;
  a.corr = corr;
  a.race = (unsigned long long*)ws;
  a.lse_part = (float2*)((char*)ws + p.race_bytes);
  a.seed_lo = (unsigned int)seed;
  a.seed_hi = (unsigned int)(seed >> 32);
  a.invT = 1.f / temperature;
  a.B = B;
  a.N = N;
  a.V = V;
  a.Dmax = Dmax;
  a.nsplit = p.nsplit;
  a.nrace = p.nrace;
  a.eps = p.eps;
  a.rps = p.rps;
  return f32 ? launch_sample_t<true>(a, p, vec, st) : launch_sample_t<false>(a, p, vec, st);
}

}  // namespace tv
