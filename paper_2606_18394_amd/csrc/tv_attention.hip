// Tree-verification attention for CDNA4 (gfx950).
//
// Computes, for every draft-tree node v of every sequence and every query
// head, softmax(q_v K^T * scale + M_v) V over the sequence's cached prefix
// and the tree nodes, where the tree-causal mask M_v keeps only v's
// ancestors and v itself (Sec. 2.2, tree-causal mask and masked attention
// equations).  The ancestor relation is rebuilt inside each workgroup as a
// bitmask in LDS from the parent array; no dense mask ever exists (App. E).
//
// Work decomposition (one workgroup = 4 wave64s):
//   * rows of one (sequence b, KV head g) pair are the N*G (node, head in
//     group) pairs; a workgroup takes RB consecutive rows;
//   * the keys are cut into 32-key tiles: ceil(kv_len/32) cache tiles, then
//     the tree tiles up to the last node of the row block (a node never sees
//     a later node since parents precede children);
//   * the tiles are split into S contiguous ranges (split-KV); inside a
//     workgroup the 4 waves take every 4th tile, each with all RB rows, so
//     every K/V byte is read from memory once per workgroup.
// Per 32-key step a wave computes S^T = K Q^T with v_mfma_f32_16x16x32_bf16
// (keys on the M side, rows on the N side), runs an fp32 online softmax in
// base 2 on the accumulators, and accumulates O^T += V^T P^T, where P^T is
// taken straight from the S^T accumulators (the 32 keys of one step are
// ordered so the B operand needs no data movement) and V^T comes from LDS
// with ds_read_b64_tr_b16 transposing reads.  The 4 waves merge their
// (max, sum, O) in LDS; with S > 1 a second kernel merges the splits.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tv_plan.h"

namespace tv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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
  int B, N, Hq, Hkv, Lmax, G, M, nRB, S, nwork;
  float c;  // scale * log2(e): scores live in base-2 exponent units
};

__device__ __forceinline__ float wave_max_across_groups(float v) {
  v = fmaxf(v, __shfl_xor(v, 16));
  v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ float wave_sum_across_groups(float v) {
  v += __shfl_xor(v, 16);
  v += __shfl_xor(v, 32);
  return v;
}

__device__ __forceinline__ void decode_work(const AttnArgs& a, int& b, int& g,
                                            int& rb, int& s) {
  // Consecutive work items (all row blocks and splits of one (b, g) pair)
  // go to the same XCD: workgroups are dispatched round-robin over the 8
  // XCDs, so item w runs on XCD w / per.
  const int per = gridDim.x / kXcds;
  int w = (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
  s = w % a.S;
  w /= a.S;
  rb = w % a.nRB;
  w /= a.nRB;
  g = w % a.Hkv;
  b = w / a.Hkv;
}

template <int D, int RB>
__global__ __launch_bounds__(256, 1) void attn_main(AttnArgs a) {
  constexpr int NT = RB / 16;        // 16-row tiles
  constexpr int NC = D / 32;         // 32-wide head-dim chunks (QK^T)
  constexpr int DT = D / 16;         // 16-wide head-dim tiles (PV)
  constexpr int CPR = D / 8;         // 16-byte chunks per K/V row
  constexpr int VL = kKeyTile * CPR / 64;  // V chunks per lane per step
  constexpr int VS = D * 2 + 32;     // LDS row stride of the V tile, bytes
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

  {
    const int per = gridDim.x / kXcds;
    const int w = (blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
    if (w >= a.nwork) return;
  }
  int b, g, rb, s;
  decode_work(a, b, g, rb, s);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;

  int kvl = a.kv_len ? a.kv_len[b] : a.Lmax;
  kvl = kvl < 0 ? 0 : (kvl > a.Lmax ? a.Lmax : kvl);
  const int r0 = rb * RB;
  const int rows = min(RB, a.M - r0);
  const int i_lo = r0 / a.G, i_hi = (r0 + rows - 1) / a.G;
  const int nct = (kvl + kKeyTile - 1) / kKeyTile;
  const int ntt = i_hi / kKeyTile + 1;
  const int T = nct + ntt;
  const int per_split = (T + a.S - 1) / a.S;
  const int t0 = s * per_split;
  const int t1 = min(T, t0 + per_split);
  const bool has_tree = t1 > nct;

  unsigned char* vbuf = smem + (size_t)wave * kKeyTile * VS;
  uint32_t* anc = reinterpret_cast<uint32_t*>(smem + (size_t)kWaves * kKeyTile * VS);
  const int anc_nodes = RB / a.G + 2;
  int32_t* par = reinterpret_cast<int32_t*>(anc + anc_nodes * ntt);
  int* flag = par + a.N;

  const size_t cache_base = (size_t)b * a.Lmax * a.Hkv * D + (size_t)g * D;
  const size_t tree_base = (size_t)b * a.N * a.Hkv * D + (size_t)g * D;
  const size_t krow = (size_t)a.Hkv * D;  // elements between consecutive keys

  // Element offset of key kk (0..31) of tile t, and whether it is a tree key.
  // Keys past the valid range are clamped onto a valid row; the mask zeroes
  // their weight, so clamping only keeps the reads inside the tensors.
  auto key_row = [&](int t, int kk, bool& tree) -> size_t {
    if (t < nct) {
      int k = t * kKeyTile + kk;
      k = k < kvl ? k : kvl - 1;
      tree = false;
      return cache_base + (size_t)k * krow;
    }
    int u = (t - nct) * kKeyTile + kk;
    u = u <= i_hi ? u : i_hi;
    tree = true;
    return tree_base + (size_t)u * krow;
  };

  // ---- queries: B operand of S^T = K Q^T, lane holds Q[row l16][8*g4 .. +8]
  bf16x8 qf[NT][NC];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = r0 + nt * 16 + l16;
    const bool ok = r < a.M;
    const int node = ok ? r / a.G : 0;
    const int h = g * a.G + (ok ? r % a.G : 0);
    const __bf16* qp = a.q + ((size_t)(b * a.N + node) * a.Hq + h) * D + 8 * g4;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      bf16x8 v = *reinterpret_cast<const bf16x8*>(qp + 32 * c);
      if (!ok) v = bf16x8{};
      qf[nt][c] = v;
    }
  }

  // ---- tree structure: ancestor-or-self bitmask of this block's nodes
  if (has_tree) {
    int bad = 0;
    for (int i = tid; i < a.N; i += 256) {
      const int p = a.parent[(size_t)b * a.N + i];
      par[i] = p;
      bad |= (i == 0) ? (p != -1) : (p < 0 || p >= i);
    }
    bad = __syncthreads_or(bad);
    const int nodes = i_hi - i_lo + 1;
    for (int t = tid; t < nodes; t += 256) {
      uint32_t* w = anc + t * ntt;
      for (int k = 0; k < ntt; ++k) w[k] = 0u;
      int u = i_lo + t;
      for (;;) {
        w[u >> 5] |= 1u << (u & 31);
        if (u == 0) break;
        const int p = par[u];
        if (p < 0 || p >= u) break;  // invalid tree: output becomes NaN
        u = p;
      }
    }
    if (tid == 0) *flag = bad;
    __syncthreads();
  }

  f32x4 o[DT][NT];
  float m[NT], lsum[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m[nt] = -INFINITY;
    lsum[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // K fragments (A operand of S^T): lane holds K[key 16*tt + l16][32c + 8*g4 ..]
  bf16x8 kn[2][NC];
  // V chunks staged through registers: chunk lane + 64*j of the 32 x D tile
  bf16x8 vn[VL];
  auto load_tile = [&](int t) {
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      bool tree;
      const size_t off = key_row(t, 16 * tt + l16, tree) + 8 * g4;
      const __bf16* kp = (tree ? a.kt : a.kc) + off;
#pragma unroll
      for (int c = 0; c < NC; ++c) kn[tt][c] = *reinterpret_cast<const bf16x8*>(kp + 32 * c);
    }
#pragma unroll
    for (int j = 0; j < VL; ++j) {
      const int id = lane + 64 * j;
      bool tree;
      const size_t off = key_row(t, id / CPR, tree) + 8 * (id % CPR);
      vn[j] = *reinterpret_cast<const bf16x8*>((tree ? a.vt : a.vc) + off);
    }
  };

  int t = t0 + wave;
  if (t < t1) load_tile(t);
  for (; t < t1; t += kWaves) {
    // stage V of tile t into this wave's LDS tile (row-major, padded rows)
#pragma unroll
    for (int j = 0; j < VL; ++j) {
      const int id = lane + 64 * j;
      *reinterpret_cast<bf16x8*>(vbuf + (id / CPR) * VS + (id % CPR) * 16) = vn[j];
    }
    bf16x8 kc[2][NC];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int c = 0; c < NC; ++c) kc[tt][c] = kn[tt][c];
    const int tn = t + kWaves;
    if (tn < t1) load_tile(tn);

    // S^T tile: lane holds S^T[key 16*tt + 4*g4 + j][row 16*nt + l16]
    f32x4 sc[2][NT];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc[tt][c], qf[nt][c], acc, 0, 0, 0);
        sc[tt][nt] = acc;
      }

    // masks: the cache tail and the tree tiles
    if (t < nct) {
      if ((t + 1) * kKeyTile > kvl) {
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const bool vis = t * kKeyTile + 16 * tt + 4 * g4 + j < kvl;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              if (!vis) sc[tt][nt][j] = -INFINITY;
          }
      }
    } else {
      const int word = t - nct;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int r = r0 + nt * 16 + l16;
        int node = (r < a.M ? r : a.M - 1) / a.G - i_lo;
        const uint32_t bits = anc[node * ntt + word];
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (!((bits >> (16 * tt + 4 * g4 + j)) & 1u)) sc[tt][nt][j] = -INFINITY;
      }
    }

    // online softmax (base 2) and the bf16 P^T operand
    bf16x8 pf[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float mx = fmaxf(fmaxf(fmaxf(sc[0][nt][0], sc[0][nt][1]), fmaxf(sc[0][nt][2], sc[0][nt][3])),
                       fmaxf(fmaxf(sc[1][nt][0], sc[1][nt][1]), fmaxf(sc[1][nt][2], sc[1][nt][3])));
      mx = wave_max_across_groups(mx) * a.c;
      const float mnew = fmaxf(m[nt], mx);
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(m[nt] - mref);
      m[nt] = mnew;
      float ps = 0.f;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = __builtin_amdgcn_exp2f(fmaf(sc[tt][nt][j], a.c, -mref));
          ps += p;
          pf[nt][4 * tt + j] = (__bf16)p;
        }
      lsum[nt] = lsum[nt] * alpha + ps;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt][nt] *= alpha;
    }

    // O^T += V^T P^T; the transposing reads give lane (g4, l16) the values
    // V[key 4*g4 + j (+16)][16*dt + l16], matching the key order of P^T
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const unsigned char* src = vbuf + (4 * g4 + (l16 >> 2)) * VS + (16 * dt + 4 * (l16 & 3)) * 2;
      typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src));
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src + 16 * VS));
      const bf16x4 lob = __builtin_bit_cast(bf16x4, lo), hib = __builtin_bit_cast(bf16x4, hi);
      const bf16x8 vf = {lob[0], lob[1], lob[2], lob[3], hib[0], hib[1], hib[2], hib[3]};
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        o[dt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[nt], o[dt][nt], 0, 0, 0);
    }
  }

  // ---- merge the 4 waves (each saw a disjoint subset of this range's keys)
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) lsum[nt] = wave_sum_across_groups(lsum[nt]);
  const int invalid = has_tree ? *flag : 0;
  __syncthreads();  // V staging and tree tables are dead from here on
  f32x4* obuf = reinterpret_cast<f32x4*>(smem);
  float2* mlbuf = reinterpret_cast<float2*>(smem + (size_t)kWaves * RB * D * 4);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) obuf[((wave * DT + dt) * NT + nt) * 64 + lane] = o[dt][nt];
  if (g4 == 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) mlbuf[wave * RB + nt * 16 + l16] = make_float2(m[nt], lsum[nt]);
  }
  __syncthreads();

  const int bg = b * a.Hkv + g;
  for (int f = wave; f < DT * NT; f += kWaves) {
    const int dt = f / NT, nt = f % NT;
    const int row = nt * 16 + l16;
    float mw[kWaves], mstar = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      mw[w] = mlbuf[w * RB + row].x;
      mstar = fmaxf(mstar, mw[w]);
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float l = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float e = mw[w] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw[w] - mstar);
      l += e * mlbuf[w * RB + row].y;
      acc += e * obuf[((w * DT + dt) * NT + nt) * 64 + lane];
    }
    if (a.S == 1) {
      const int r = r0 + row;
      if (r < a.M) {
        const int node = r / a.G, h = g * a.G + r % a.G;
        const float inv = invalid ? NAN : 1.f / l;
        bf16x4 ov = {(__bf16)(acc[0] * inv), (__bf16)(acc[1] * inv), (__bf16)(acc[2] * inv),
                     (__bf16)(acc[3] * inv)};
        *reinterpret_cast<bf16x4*>(a.out + ((size_t)(b * a.N + node) * a.Hq + h) * D + 16 * dt +
                                   4 * g4) = ov;
      }
    } else {
      const size_t fr = ((size_t)(bg * a.nRB + rb) * a.S + s) * DT * NT;
      a.ws_o[(fr + dt * NT + nt) * 64 + lane] = acc;
      if (dt == 0 && g4 == 0)
        a.ws_ml[((size_t)(bg * a.nRB + rb) * a.S + s) * RB + row] = make_float2(mstar, l);
    }
  }
}

// Merge the S key-range partials of every row: out = sum_s e_s O_s /
// sum_s e_s l_s with e_s = 2^(m_s - max m).  One wave per 16x16 fragment.
template <int D, int RB>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
  constexpr int NT = RB / 16, DT = D / 16;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g4 = lane >> 4, l16 = lane & 15;
  const int F = blockIdx.x * 4 + wave;       // fragment id, all 4 in one (b,g,rb)
  const int per_blk = DT * NT;
  const int blk = F / per_blk, f = F % per_blk;
  const int rb = blk % a.nRB, bg = blk / a.nRB;
  const int b = bg / a.Hkv, g = bg % a.Hkv;
  int bad = 0;
  for (int i = threadIdx.x; i < a.N; i += 256) {
    const int p = a.parent[(size_t)b * a.N + i];
    bad |= (i == 0) ? (p != -1) : (p < 0 || p >= i);
  }
  bad = __syncthreads_or(bad);
  const int dt = f / NT, nt = f % NT;
  const int row = nt * 16 + l16, r = rb * RB + row;
  if (r >= a.M) return;
  const size_t base = (size_t)(bg * a.nRB + rb) * a.S;
  float mstar = -INFINITY;
  for (int s = 0; s < a.S; ++s) mstar = fmaxf(mstar, a.ws_ml[(base + s) * RB + row].x);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float l = 0.f;
  for (int s = 0; s < a.S; ++s) {
    const float2 ml = a.ws_ml[(base + s) * RB + row];
    if (ml.x == -INFINITY) continue;
    const float e = __builtin_amdgcn_exp2f(ml.x - mstar);
    l += e * ml.y;
    acc += e * a.ws_o[((base + s) * DT * NT + dt * NT + nt) * 64 + lane];
  }
  const float inv = bad ? NAN : 1.f / l;
  const int node = r / a.G, h = g * a.G + r % a.G;
  bf16x4 ov = {(__bf16)(acc[0] * inv), (__bf16)(acc[1] * inv), (__bf16)(acc[2] * inv),
               (__bf16)(acc[3] * inv)};
  *reinterpret_cast<bf16x4*>(a.out + ((size_t)(b * a.N + node) * a.Hq + h) * D + 16 * dt + 4 * g4) = ov;
}

template <int D, int RB>
static hipError_t launch_attn_t(const AttnArgs& a, const AttnPlan& p, hipStream_t st) {
  hipError_t e0 = hipFuncSetAttribute((const void*)attn_main<D, RB>,
                                      hipFuncAttributeMaxDynamicSharedMemorySize,
                                      (int)p.lds_bytes);
  if (e0 != hipSuccess) return e0;
  hipLaunchKernelGGL((attn_main<D, RB>), dim3(p.grid), dim3(256), p.lds_bytes, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.S == 1) return e;
  const int frags = a.B * a.Hkv * p.nRB * (D / 16) * (RB / 16);
  hipLaunchKernelGGL((attn_combine<D, RB>), dim3(frags / 4), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attention(const void* q, const void* kc, const void* vc, const void* kt,
                            const void* vt, const int32_t* parent, const int32_t* kv_len,
                            void* out, int B, int N, int Hq, int Hkv, int D, int Lmax,
                            float scale, void* ws, const AttnPlan& p, hipStream_t st) {
  AttnArgs a;
  a.q = (const __bf16*)q;
  a.kc = (const __bf16*)kc;
  a.vc = (const __bf16*)vc;
  a.kt = (const __bf16*)kt;
  a.vt = (const __bf16*)vt;
  a.parent = parent;
  a.kv_len = kv_len;
  a.out = (__bf16*)out;
  a.ws_o = (f32x4*)ws;
  a.ws_ml = (float2*)((char*)ws + p.ws_o_bytes);
  a.B = B;
  a.N = N;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.Lmax = Lmax;
  a.G = p.G;
  a.M = p.M;
  a.nRB = p.nRB;
  a.S = p.S;
  a.nwork = p.nwork;
  a.c = scale * 1.4426950408889634f;
  if (D == 128) return p.RB == 64 ? launch_attn_t<128, 64>(a, p, st) : launch_attn_t<128, 32>(a, p, st);
  return p.RB == 64 ? launch_attn_t<64, 64>(a, p, st) : launch_attn_t<64, 32>(a, p, st);
}

}  // namespace tv
