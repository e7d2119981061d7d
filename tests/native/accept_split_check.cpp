// Host check of the acceptance scan's split count (tv_plan.h): for each
// "B N V esize" on stdin, prints the planned splits, the workgroup count and
// the share of load slots the split uses, so the caller can compare them
// with the rule: among the counts from the ~2048-workgroup target down to
// half of it, the one using the largest share of its slots.
#include <cstdio>
#include "tv_plan.h"

int main() {
  int B, N, V, esize;
  while (std::scanf("%d %d %d %d", &B, &N, &V, &esize) == 4) {
    const int vec = 16 / esize;
    const tv::AcceptPlan p = tv::accept_plan(B, N, V, esize, vec);
    const long long chunks = ((long long)V + vec - 1) / vec;
    const long long per_round = (long long)tv::kAcceptScanThreads * tv::kAcceptScanLoads;
    std::printf("%d %d %d %d %d %.4f\n", B, N, V, esize, p.nsplit,
                tv::accept_round_fill(chunks, p.nsplit, per_round));
  }
  return 0;
}
