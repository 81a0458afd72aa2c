// Host-only check of the decision-pass workspace bounds: for each input line
// "V B_max rows_max", every plan of b <= B_max sequences and u <= rows_max
// rows must fit vocab_ws_bound / tree_ws_bound, and every draft plan of
// n <= B_max rows draft_ws_bound.  Prints "ok" or the first plan that does
// not fit.
#include <cstdio>

#include "vocab.h"

int main() {
  int V, B, N;
  while (std::scanf("%d %d %d", &V, &B, &N) == 3) {
    const size_t vb = spec::vocab_ws_bound(B, N), tb = spec::tree_ws_bound(B, N), db = spec::draft_ws_bound(B);
    bool ok = true;
    for (int b = 1; b <= B && ok; ++b) {
      const size_t d = spec::draft_ws_bytes(spec::draft_plan(b, V));
      if (d > db) {
        std::printf("draft V=%d n=%d %zu > %zu\n", V, b, d, db);
        ok = false;
      }
      for (int u = b; u <= N && ok; ++u) {
        const spec::VocabPlan p = spec::vocab_plan(b, u, V);
        if (spec::vocab_ws_bytes(p) > vb || spec::tree_ws_bytes(p) > tb) {
          std::printf("vocab V=%d B=%d rows=%d %zu/%zu > %zu/%zu\n", V, b, u, spec::vocab_ws_bytes(p),
                      spec::tree_ws_bytes(p), vb, tb);
          ok = false;
        }
      }
    }
    if (ok) std::printf("ok\n");
  }
  return 0;
}
