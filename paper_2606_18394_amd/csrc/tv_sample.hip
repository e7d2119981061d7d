// Non-greedy tree acceptance (temperature T > 0) for CDNA4 (gfx950): the
// speculative sampling test of every draft node, the deepest accepted path,
// and the correction token drawn at its last node (Sec. 2.4).
//
// With p_u = softmax(logits[u] / T) and q_d = softmax(draft_logits[d-1] / T),
// draft node i (token y, parent u, depth d) passes when
// u_i * q_d(y) < p_u(y), i.e. u_i < min(1, p/q); it is accepted when it
// passes and its parent is accepted.  The correction token at the deepest
// accepted node v comes from max(0, p_v - q_{d(v)+1}) when v has children
// (all of them rejected), else from p_v (an all-zero residual falls back to
// p_v too), by an exponential race: the winner is argmax w(x) / E_x with
// E_x = -ln U(b, x), U from Philox4x32-10 (Salmon et al., SC 2011) on the
// counter (x / 4, b, 0, 0) and the 64-bit seed as key, word x % 4, mapped
// to (0, 1) by its top 23 bits.
//
// Three kernels:
//   lse_scan: one workgroup per (row, vocabulary split) over the B*N target
//     rows and the B*Nd draft rows: running (max, sum of exponentials) of
//     x / T per thread, merged across the workgroup.
//   sample_accept: one workgroup per (sequence, vocabulary split).  Each
//     merges the log-sum-exps of its sequence, runs the acceptance (depths,
//     then the root-path AND of the tests, both by pointer jumping) and
//     races its vocabulary slice for the correction token, keeping two
//     keys: the residual race and the plain p_v race.  Split 0 writes the
//     path.  Every workgroup of a sequence repeats the acceptance, which
//     costs less than a kernel boundary between acceptance and race.
//   sample_finish: one wave per sequence merges the race keys.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv_plan.h"

namespace tv {

struct SampleArgs {
  const void* logits;   // [B, N, V] target
  const void* dlogits;  // [B, Nd, V] draft head, row d - 1 = depth d
  const int32_t* draft;
  const int32_t* parent;
  const float* u;       // [B, N] acceptance uniforms
  int32_t* accept_len;
  int32_t* path;
  int32_t* corr;
  unsigned long long* race;  // [B, nrace, 2] race keys
  float2* lse_part;          // [B*N + B*Nd, nsplit] (max, sum exp) of x / T
  unsigned int seed_lo, seed_hi;
  float invT;
  int B, N, V, Nd, Dmax, nsplit, nrace;
  long long eps;  // vocabulary entries per lse split, a multiple of 8
  long long rps;  // vocabulary entries per race split, a multiple of 8
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

__device__ __forceinline__ unsigned long long wave_max_key(unsigned long long k) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const unsigned int lo = __shfl_xor((unsigned int)k, o);
    const unsigned int hi = __shfl_xor((unsigned int)(k >> 32), o);
    const unsigned long long other = ((unsigned long long)hi << 32) | lo;
    k = other > k ? other : k;
  }
  return k;
}

// ------------------------------------------------------------ lse_scan

// (max, sum exp) of x / T over elements [x0, x1) of a row; x0 and x1 are
// multiples of 8 (or x1 = V) so that vectorised rows read whole 16-byte
// chunks of either dtype
template <bool F32>
__device__ __forceinline__ void lse_slice(const void* rowp, long long x0, long long x1, bool vec,
                                          float invT, float& m, float& s) {
  constexpr int E = F32 ? 4 : 8;  // elements per 16-byte chunk
  constexpr int L = kScanLoadsPerThread;
  const int tid = threadIdx.x;
  if (vec) {
    const long long c0 = x0 / E, c1 = (x1 + E - 1) / E;
    const uint4* base = reinterpret_cast<const uint4*>(rowp);
    for (long long c = c0 + tid; c < c1; c += (long long)L * kScanThreads) {
      // all L loads are issued first (past the end: the last chunk again),
      // then decoded with the padding replaced by -inf bit patterns, so the
      // loads are in flight together
      constexpr unsigned int kNegInf = F32 ? 0xFF800000u : 0xFF80FF80u;
      uint4 raw[L];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const long long cu = c + (long long)u * kScanThreads;
        raw[u] = base[cu < c1 ? cu : c1 - 1];
      }
      float x[L][E];
#pragma unroll
      for (int u = 0; u < L; ++u) {
        const bool in = c + (long long)u * kScanThreads < c1;
        const unsigned int ws[4] = {in ? raw[u].x : kNegInf, in ? raw[u].y : kNegInf,
                                    in ? raw[u].z : kNegInf, in ? raw[u].w : kNegInf};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (F32) {
            x[u][k] = __uint_as_float(ws[k]) * invT;
          } else {
            x[u][2 * k] = __uint_as_float(ws[k] << 16) * invT;
            x[u][2 * k + 1] = __uint_as_float(ws[k] & 0xFFFF0000u) * invT;
          }
        }
      }
      float bm = -INFINITY;
#pragma unroll
      for (int u = 0; u < L; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) bm = fmaxf(bm, x[u][e]);
      if (bm == -INFINITY) continue;
      const float mn = fmaxf(m, bm);
      float bs = 0.f;
#pragma unroll
      for (int u = 0; u < L; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) bs += __expf(x[u][e] - mn);
      s = (m == -INFINITY ? 0.f : s * __expf(m - mn)) + bs;
      m = mn;
    }
  } else {
    for (long long c = x0 + tid; c < x1; c += kScanThreads) {
      const float x = load_logit<F32>(rowp, (size_t)c) * invT;
      lse_merge2(m, s, x, 1.f);
    }
  }
}

template <bool F32T, bool F32D>
__global__ __launch_bounds__(kScanThreads) void lse_scan(SampleArgs a, int vec) {
  const int row = blockIdx.x / a.nsplit, split = blockIdx.x % a.nsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int trows = a.B * a.N;
  const long long x0 = (long long)split * a.eps;
  const long long x1 = x0 + a.eps < a.V ? x0 + a.eps : a.V;
  float m = -INFINITY, s = 0.f;
  if (row < trows) {
    const char* rowp = (const char*)a.logits + (size_t)row * a.V * (F32T ? 4 : 2);
    lse_slice<F32T>(rowp, x0, x1, vec != 0, a.invT, m, s);
  } else {
    const char* rowp = (const char*)a.dlogits + (size_t)(row - trows) * a.V * (F32D ? 4 : 2);
    lse_slice<F32D>(rowp, x0, x1, vec != 0, a.invT, m, s);
  }
  __shared__ float rm[kScanThreads / 64], rs[kScanThreads / 64];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) lse_merge2(m, s, __shfl_xor(m, o), __shfl_xor(s, o));
  if (lane == 0) {
    rm[wave] = m;
    rs[wave] = s;
  }
  __syncthreads();
  if (tid == 0) {
    float gm = rm[0], gs = rs[0];
#pragma unroll
    for (int w = 1; w < kScanThreads / 64; ++w) lse_merge2(gm, gs, rm[w], rs[w]);
    a.lse_part[(size_t)row * a.nsplit + split] = make_float2(gm, gs);
  }
}

// ------------------------------------------------------------ sample_accept

constexpr int kSampleThreads = 512;
constexpr int kNodesPerThread = kMaxNodes / kSampleThreads;

template <bool F32T, bool F32D>
__global__ __launch_bounds__(kSampleThreads) void sample_accept(SampleArgs a, int vec) {
  __shared__ float lse_t[kMaxNodes];
  __shared__ float lse_d[kMaxDraftDepth];
  __shared__ short par[kMaxNodes], jmp0[kMaxNodes], jmp1[kMaxNodes], dep0[kMaxNodes],
      dep1[kMaxNodes];
  __shared__ unsigned char ok0[kMaxNodes], ok1[kMaxNodes];
  __shared__ unsigned int best_key;
  __shared__ unsigned long long red[2][kSampleThreads / 64];

  const int b = blockIdx.x / a.nrace, sp = blockIdx.x % a.nrace;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.N, Nd = a.Nd, V = a.V;

  // ---- tree, tokens, log-sum-exps
  int bad = 0;
  int tok[kNodesPerThread];
#pragma unroll
  for (int k = 0; k < kNodesPerThread; ++k) {
    const int i = tid + kSampleThreads * k;
    tok[k] = 0;
    if (i < N) {
      const int p = a.parent[(size_t)b * N + i];
      const int badi = (i == 0) ? (p != -1) : (p < 0 || p >= i);
      bad |= badi;
      par[i] = (short)(badi || i == 0 ? 0 : p);
      tok[k] = a.draft[(size_t)b * N + i];
    }
  }
  for (int r = tid; r < N + Nd; r += kSampleThreads) {
    const size_t row = r < N ? (size_t)b * N + r : (size_t)a.B * N + (size_t)b * Nd + (r - N);
    float m = -INFINITY, s = 0.f;
    for (int k = 0; k < a.nsplit; ++k) {
      const float2 ps = a.lse_part[row * a.nsplit + k];
      lse_merge2(m, s, ps.x, ps.y);
    }
    const float l = m + __logf(s);
    if (r < N) lse_t[r] = l;
    else lse_d[r - N] = l;
  }
  if (tid == 0) best_key = 0u;
  bad = __syncthreads_or(bad);

  int len = -1, v = 0, dv = 0;
  if (!bad && N <= 64) {
    // Trees of at most 64 nodes: wave 0 alone, lane i holding node i, with
    // lane exchanges in place of LDS rounds and workgroup barriers.  Every
    // lane of the wave takes part in each exchange.
    __shared__ int s_res[3];
    if (wave == 0) {
      const int i = lane;
      const bool node = i < N;
      const int pp = node && i > 0 ? par[i] : 0;  // the root jumps to itself
      int jmp = pp, dep = node && i > 0 ? 1 : 0;
      for (int r = 0; r < 6 && __any(jmp != 0); ++r) {
        dep += __shfl(dep, jmp);
        jmp = __shfl(jmp, jmp);
      }
      const bool deep = __any(node && dep > Nd);
      int ok = node ? 1 : 0;
      if (node && i > 0 && dep <= Nd) {
        const int y = tok[0];
        ok = 0;
        if (y >= 0 && y < V) {
          const float pl = load_logit<F32T>(a.logits, ((size_t)b * N + pp) * V + y);
          const float ql = load_logit<F32D>(a.dlogits, ((size_t)b * Nd + dep - 1) * V + y);
          const float p = __expf(pl * a.invT - lse_t[pp]);
          const float q = __expf(ql * a.invT - lse_d[dep - 1]);
          ok = a.u[(size_t)b * N + i] * q < p;
        }
      }
      jmp = pp;
      for (int r = 0; r < 6 && __any(jmp != 0); ++r) {
        ok &= __shfl(ok, jmp);
        jmp = __shfl(jmp, jmp);
      }
      unsigned int k = ok ? ((unsigned int)dep << 16) | (0xFFFFu - (unsigned int)i) : 0u;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        const unsigned int other = __shfl_xor(k, o);
        k = other > k ? other : k;
      }
      if (lane == 0) {
        const int d = (int)(k >> 16);
        s_res[0] = deep || d + 1 > a.Dmax ? -1 : d + 1;
        s_res[1] = (int)(0xFFFFu - (k & 0xFFFFu));
        s_res[2] = d;
      }
    }
    __syncthreads();
    len = s_res[0];
    v = s_res[1];
    dv = s_res[2];
  } else if (!bad) {
    // depths by pointer jumping (the root jumps to itself)
    for (int i = tid; i < N; i += kSampleThreads) {
      jmp0[i] = par[i];
      dep0[i] = i == 0 ? 0 : 1;
    }
    __syncthreads();
    int cur = 0, more, rounds = 0;
    do {
      const short* jc = cur ? jmp1 : jmp0;
      const short* dc = cur ? dep1 : dep0;
      short* jn = cur ? jmp0 : jmp1;
      short* dn = cur ? dep0 : dep1;
      more = 0;
      for (int i = tid; i < N; i += kSampleThreads) {
        const int j = jc[i];
        dn[i] = dc[i] + dc[j];
        jn[i] = jc[j];
        more |= jc[j] != 0;
      }
      cur ^= 1;
    } while (__syncthreads_or(more) && ++rounds < 16);
    const short* depth = cur ? dep1 : dep0;
    // the test of every node, then the AND over its root path
    int deep = 0;
#pragma unroll
    for (int k = 0; k < kNodesPerThread; ++k) {
      const int i = tid + kSampleThreads * k;
      if (i >= N) break;
      const int d = depth[i];
      deep |= d > Nd;
      unsigned char t = 1;
      if (i > 0 && d <= Nd) {
        const int y = tok[k], u = par[i];
        t = 0;
        if (y >= 0 && y < V) {
          const float pl = load_logit<F32T>(a.logits, ((size_t)b * N + u) * V + y);
          const float ql = load_logit<F32D>(a.dlogits, ((size_t)b * Nd + d - 1) * V + y);
          const float p = __expf(pl * a.invT - lse_t[u]);
          const float q = __expf(ql * a.invT - lse_d[d - 1]);
          t = a.u[(size_t)b * N + i] * q < p;
        }
      }
      ok0[i] = t;
      jmp0[i] = par[i];
    }
    bad = __syncthreads_or(deep);  // deeper than the draft logits reach
    if (!bad) {
      cur = 0;
      rounds = 0;
      do {
        const short* jc = cur ? jmp1 : jmp0;
        const unsigned char* oc = cur ? ok1 : ok0;
        short* jn = cur ? jmp0 : jmp1;
        unsigned char* on = cur ? ok0 : ok1;
        more = 0;
        for (int i = tid; i < N; i += kSampleThreads) {
          const int j = jc[i];
          on[i] = oc[i] & oc[j];
          jn[i] = jc[j];
          more |= jc[j] != 0;
        }
        cur ^= 1;
      } while (__syncthreads_or(more) && ++rounds < 16);
      const unsigned char* acc = cur ? ok1 : ok0;
      unsigned int mk = 0u;
      for (int i = tid; i < N; i += kSampleThreads)
        if (acc[i]) {
          const unsigned int k = ((unsigned int)depth[i] << 16) | (0xFFFFu - (unsigned int)i);
          mk = mk > k ? mk : k;
        }
      atomicMax(&best_key, mk);
      __syncthreads();
      const unsigned int bk = best_key;
      dv = (int)(bk >> 16);
      v = (int)(0xFFFFu - (bk & 0xFFFFu));
      len = dv + 1 > a.Dmax ? -1 : dv + 1;
    }
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

  // ---- the race over this split's slice of the vocabulary
  int child = 0;
  for (int i = 1 + tid; i < N; i += kSampleThreads) child |= par[i] == v;
  const bool has_child = __syncthreads_or(child) != 0;
  const float lv = lse_t[v];
  const float lq = has_child ? lse_d[dv] : 0.f;
  const size_t prow = ((size_t)b * N + v) * V;
  const size_t qrow = ((size_t)b * Nd + dv) * V;
  const long long x0 = (long long)sp * a.rps;
  const long long x1 = x0 + a.rps < V ? x0 + a.rps : V;
  unsigned long long kres = 0ull, kp = 0ull;
  for (long long xg = x0 + 8ll * tid; xg < x1; xg += 8ll * kSampleThreads) {
    float pl[8], ql[8];
    if (vec && xg + 8 <= x1) {
      load8<F32T>(a.logits, prow + xg, pl);
      if (has_child) load8<F32D>(a.dlogits, qrow + xg, ql);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pl[e] = xg + e < x1 ? load_logit<F32T>(a.logits, prow + xg + e) : -INFINITY;
        ql[e] = has_child && xg + e < x1 ? load_logit<F32D>(a.dlogits, qrow + xg + e) : 0.f;
      }
    }
    const uint4 r0 = philox4x32_10(make_uint4((unsigned int)(xg >> 2), (unsigned int)b, 0u, 0u),
                                   a.seed_lo, a.seed_hi);
    const uint4 r1 = philox4x32_10(
        make_uint4((unsigned int)(xg >> 2) + 1u, (unsigned int)b, 0u, 0u), a.seed_lo, a.seed_hi);
    const unsigned int words[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (xg + e >= x1) break;
      const float inv_e = 1.f / -__logf(open_uniform(words[e]));
      const float p = __expf(pl[e] * a.invT - lv);
      const unsigned int x = (unsigned int)(xg + e);
      if (p > 0.f) {
        const unsigned long long k = race_key(p * inv_e, x);
        kp = k > kp ? k : kp;
      }
      if (has_child) {
        const float w = p - __expf(ql[e] * a.invT - lq);
        if (w > 0.f) {
          const unsigned long long k = race_key(w * inv_e, x);
          kres = k > kres ? k : kres;
        }
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
    const unsigned long long k = kres ? kres : kp;  // all-zero residual: race on p
    a.corr[b] = a.accept_len[b] < 0 || k == 0ull ? -1 : (int)(0xFFFFFFFFu - (unsigned int)k);
  }
}

// ------------------------------------------------------------ launch

template <bool F32T, bool F32D>
static hipError_t launch_sample_t(const SampleArgs& a, const SamplePlan& p, int vec,
                                  hipStream_t st) {
  hipLaunchKernelGGL((lse_scan<F32T, F32D>), dim3(p.lse_grid), dim3(kScanThreads), 0, st, a, vec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((sample_accept<F32T, F32D>), dim3(a.B * p.nrace), dim3(kSampleThreads), 0,
                     st, a, vec);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(sample_finish, dim3(a.B), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sample(const void* logits, int f32t, const void* dlogits, int f32d,
                         const int32_t* draft, const int32_t* parent, const float* u,
                         unsigned long long seed, float temperature, int B, int N, int V, int Nd,
                         int Dmax, int32_t* accept_len, int32_t* path, int32_t* corr, void* ws,
                         hipStream_t st) {
  const SamplePlan p = sample_plan(B, N, V, Nd);
  const int vec = (uintptr_t)logits % 16 == 0 && (uintptr_t)dlogits % 16 == 0 && V % 8 == 0;
  SampleArgs a;
  a.logits = logits;
  a.dlogits = dlogits;
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
  a.Nd = Nd;
  a.Dmax = Dmax;
  a.nsplit = p.nsplit;
  a.nrace = p.nrace;
  a.eps = p.eps;
  a.rps = p.rps;
  if (f32t) {
    return f32d ? launch_sample_t<true, true>(a, p, vec, st)
                : launch_sample_t<true, false>(a, p, vec, st);
  }
  return f32d ? launch_sample_t<false, true>(a, p, vec, st)
              : launch_sample_t<false, false>(a, p, vec, st);
}

}  // namespace tv
