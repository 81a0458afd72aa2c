// Host-only driver of the attention work planner (plan_attention): reads
// planning problems from stdin and prints each plan, for the CPU test that
// checks its invariants.  Input per problem: "G Hkv max_parts target_wgs
// allow_prefill n_segments" then n_segments lines "seq row0 nrows pos0".
// Output per problem: "plan nt w prefill n_parts n_items n_groups", then one
// line per item "item row0 nrows pos0 seq t0 t1 part" and per group
// "group row0 nrows part0 nparts".
#include <cstdio>
#include <vector>

#include "host_util.h"

int main() {
  int G, Hkv, max_parts, target_wgs, allow_prefill, n;
  while (std::scanf("%d %d %d %d %d %d", &G, &Hkv, &max_parts, &target_wgs, &allow_prefill, &n) == 6) {
    std::vector<spec::AttnSegment> segs(n);
    for (auto& s : segs)
      if (std::scanf("%d %d %d %d", &s.seq, &s.row0, &s.nrows, &s.pos0) != 4) return 1;
    const spec::AttnPlan p = spec::plan_attention(segs, G, Hkv, max_parts, target_wgs, allow_prefill != 0);
    std::printf("plan %d %d %d %d %zu %zu\n", p.nt, p.w, p.prefill ? 1 : 0, p.n_parts, p.items.size(),
                p.groups.size());
    for (const auto& it : p.items)
      std::printf("item %d %d %d %d %d %d %d\n", it.row0, it.nrows, it.pos0, it.seq, it.t0, it.t1, it.part);
    for (const auto& g : p.groups) std::printf("group %d %d %d %d\n", g.row0, g.nrows, g.part0, g.nparts);
  }
  return 0;
}
