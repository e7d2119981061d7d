// Host-side check of the launch plans (tv_plan.h is plain C++): for each
// shape on stdin ("B N Hq Hkv D Lmax V"), enumerate every launched
// workgroup exactly as the kernels decode it and verify that the decoded
// work items are in range and cover every (b, g, rb, s) once, that the
// workspace holds the largest index any workgroup writes, and that the
// dynamic LDS fits the 160 KB of a CDNA4 CU.  Prints "OK ..." or "FAIL ...".
#include <cstdio>
#include <vector>
#include "tv_plan.h"

int main() {
  int B, N, Hq, Hkv, D, Lmax, V;
  int bad = 0, cases = 0;
  while (std::scanf("%d %d %d %d %d %d %d", &B, &N, &Hq, &Hkv, &D, &Lmax, &V) == 7) {
    ++cases;
    const tv::AttnPlan p = tv::attn_plan(B, N, Hq, Hkv, D, Lmax);
    std::vector<int> seen((size_t)p.nwork, 0);
    const int tiles = tv::cdiv(Lmax, tv::kKeyTile) + tv::cdiv(N, tv::kKeyTile);
    bool ok = p.grid % tv::kXcds == 0 && p.nwork == B * Hkv * p.nRB * p.S && p.grid >= p.nwork;
    ok = ok && (long long)p.S * p.chunk >= tiles && (long long)(p.S - 1) * p.chunk < tiles;
    ok = ok && p.WR >= 1 && p.RB == tv::kRowsPerWave * p.WR && tv::attn_plan_fits(p);
    // the spread order needs every workgroup to carry a work item
    if (p.spread && (p.grid != p.nwork || tv::kXcds % Hkv != 0 || p.S % (tv::kXcds / Hkv) != 0))
      ok = false;
    int decoded = 0;
    for (int bid = 0; bid < p.grid && ok; ++bid) {
      tv::WorkItem it{};
      if (!tv::work_item(p.grid, p.nwork, p.S, p.nRB, p.spread, B, Hkv, bid, it)) continue;
      ++decoded;
      const int s = it.s, rb = it.rb, g = it.g, b = it.b;
      if (b < 0 || b >= B || g < 0 || g >= Hkv || rb < 0 || rb >= p.nRB || s < 0 || s >= p.S ||
          rb * p.RB >= p.M) {
        ok = false;
        break;
      }
      seen[(size_t)(s + p.S * (rb + p.nRB * (g + Hkv * b)))]++;
      if (p.S > 1) {
        const int DT = D / 16, NT = p.RB / 16;
        const size_t fr = ((size_t)((b * Hkv + g) * p.nRB + rb) * p.S + s) * DT * NT;
        const size_t last_o = (fr + (size_t)DT * NT - 1) * 64 + 63;
        const size_t last_ml = ((size_t)((b * Hkv + g) * p.nRB + rb) * p.S + s) * p.RB + p.RB - 1;
        if ((last_o + 1) * 16 > p.ws_o_bytes || (last_ml + 1) * 8 > p.ws_ml_bytes) ok = false;
      }
    }
    for (int v : seen) ok = ok && v == 1;
    ok = ok && decoded == p.nwork;
    if (p.S > 1) {
      // arrival counter + tree flag per row block; the workspace sections add up
      const size_t groups = (size_t)B * Hkv * p.nRB;
      if (groups > (size_t)tv::kSyncGroups || p.ws_sync_bytes != tv::kSyncBytes) ok = false;
      if (p.ws_bytes != p.ws_o_bytes + p.ws_ml_bytes + p.ws_sync_bytes) ok = false;
      // for any kv_len, the chunks that hold tiles are exactly the first
      // nval = min(S, ceil(T / chunk)) and one of them holds tree tiles
      for (int kvl : {0, 1, Lmax / 2, Lmax}) {
        if (kvl < 0 || kvl > Lmax) continue;
        const int nct = tv::cdiv(kvl, tv::kKeyTile);
        for (int rb = 0; rb < p.nRB; ++rb) {
          const int rows = p.M - rb * p.RB < p.RB ? p.M - rb * p.RB : p.RB;
          const int i_hi = (rb * p.RB + rows - 1) / p.G;
          const int T = nct + i_hi / tv::kKeyTile + 1;
          const int nval = p.S < tv::cdiv(T, p.chunk) ? p.S : tv::cdiv(T, p.chunk);
          int nonempty = 0, tree = 0;
          for (int s = 0; s < p.S; ++s) {
            const int t0 = s * p.chunk, t1 = t0 + p.chunk < T ? t0 + p.chunk : T;
            if (t0 < t1) {
              ++nonempty;
              tree += t1 > nct;
              if (s >= nval) ok = false;
            }
          }
          if (nonempty != nval || tree < 1 || nval < 1) ok = false;
        }
      }
    }
    if (p.lds_bytes > 160 * 1024) ok = false;
    // shared queries: several key groups of several waves, a grid that
    // fills every CU, and the queries' LDS counted in the kernel's
    if (p.qshare) {
      if (p.WK < 2 || p.WR < 2 || p.nwork < 256LL * p.wg_per_cu) ok = false;
      if (p.lds_bytes != tv::attn_lds_bytes(D, p.WR, p.WK, p.NS, p.G, N, true)) ok = false;
    } else if (p.NS > 0 && p.lds_bytes != tv::attn_lds_bytes(D, p.WR, p.WK, p.NS, p.G, N, false)) {
      ok = false;
    }
    for (int esize : {2, 4})
      for (int vec : {1, 16 / esize}) {
        const tv::AcceptPlan ap = tv::accept_plan(B, N, V, esize, vec);
        const long long nch = ((long long)V + vec - 1) / vec;
        if (ap.ws_bytes > tv::accept_ws_bytes(B, N)) ok = false;
        if (ap.grid != (long long)B * N * ap.nsplit) ok = false;
        if ((long long)ap.nsplit * ap.chunks_per_split < nch) ok = false;
        if ((long long)(ap.nsplit - 1) * ap.chunks_per_split >= nch) ok = false;
        if (ap.nsplit < 1 || ap.nsplit > tv::kAcceptMaxSplit) ok = false;
        if (ap.ws_bytes != (size_t)B * N * ap.nsplit * 8) ok = false;
        if (tv::accept_lds_bytes(N) + (size_t)N * 8 > 64 * 1024) ok = false;
        // draft top-W over Nd = min(N, 64) depth rows: every chunk in one
        // split, the workspace within its bound
        const int Nd = N < 64 ? N : 64;
        const tv::TopwPlan tp = tv::topw_plan(B, Nd, V, vec);
        if (tp.grid != (long long)B * Nd * tp.nsplit) ok = false;
        if ((long long)tp.nsplit * tp.chunks_per_split < nch) ok = false;
        if ((long long)(tp.nsplit - 1) * tp.chunks_per_split >= nch) ok = false;
        if (tp.nsplit < 1 || tp.nsplit > tv::kAcceptMaxSplit) ok = false;
        if (tp.ws_bytes > tv::topw_ws_bytes(B, Nd)) ok = false;
      }
    std::printf("%s B=%d N=%d Hq=%d Hkv=%d D=%d L=%d V=%d S=%d RB=%d nRB=%d grid=%d spread=%d lds=%zu ws=%zu\n",
                ok ? "OK" : "FAIL", B, N, Hq, Hkv, D, Lmax, V, p.S, p.RB, p.nRB, p.grid,
                p.spread, p.lds_bytes, p.ws_bytes);
    bad += !ok;
  }
  std::printf("%d cases, %d failed\n", cases, bad);
  return bad ? 1 : 0;
}
