// Attention work planning: query tiles and key-range splits.

#include <algorithm>

#include "host_util.h"

namespace spec {

AttnPlan plan_attention(const std::vector<AttnSegment>& segs, int G, int Hkv, int max_parts,
                        int target_wgs, bool allow_prefill) {
  AttnPlan p;
  int max_rows = 1, min_rows = 1 << 30;
  for (const auto& s : segs) {
    max_rows = std::max(max_rows, s.nrows);
    min_rows = std::min(min_rows, s.nrows);
  }
  int max_keys = 0;
  for (const auto& s : segs) max_keys = std::max(max_keys, s.pos0 + s.nrows);
  if (allow_prefill && !segs.empty() && min_rows >= kPrefillMinRows && G >= 1 && 256 % G == 0 &&
      max_keys <= kPrefillMaxKeys) {
    p.prefill = true;
    const int br = 256 / G;
    for (const auto& s : segs)
      for (int r = 0; r < s.nrows; r += br) {
        const int n = std::min(br, s.nrows - r);
        p.items.push_back(AttnItem{s.row0 + r, n, s.pos0 + r, s.seq, 0, s.pos0 + r + n, -1, 0});
      }
    // heaviest (most keys) first, so that the long blocks start in the first
    // round of workgroups
    std::stable_sort(p.items.begin(), p.items.end(),
                     [](const AttnItem& x, const AttnItem& y) { return x.t1 > y.t1; });
    return p;
  }
  // query vectors per tile: rows * G <= 16 * nt, nt in {1, 2, 4}
  const int want = std::min(max_rows * G, 64);
  p.nt = want <= 16 ? 1 : (want <= 32 ? 2 : 4);
  // One sequence (a batch-1 verify, draft step or tree verify: a few MB of
  // keys and values, latency-bound): twice the items with half the query
  // vectors each, when a row's query heads still fit the narrower tile (6
  // rows x 4 heads per KV head, head dim 128: 8.6 -> 7.6 us per layer; the
  // 15-node tree verify 4.76 -> 4.44 ms; halving the tree's tiles twice was
  // no better).  Several sequences keep the wider tiles, whose items read
  // their keys and values once for all rows.
  if (segs.size() == 1 && p.nt >= 2 && G <= 8 * p.nt) p.nt /= 2;
  p.w = p.nt >= 4 ? 2 : 4;  // waves per workgroup (LDS of the merge bounds it at nt = 4)
  const int qt = std::max(1, 16 * p.nt / G);

  struct Tile {
    int seq, row0, nrows, pos0, kend;
  };
  std::vector<Tile> tiles;
  long long total_keys = 0;
  for (const auto& s : segs) {
    for (int r = 0; r < s.nrows; r += qt) {
      const int n = std::min(qt, s.nrows - r);
      const int kend = s.pos0 + r + n;  // keys 0 .. last row's position
      tiles.push_back(Tile{s.seq, s.row0 + r, n, s.pos0 + r, kend});
      total_keys += kend;
    }
  }
  // key range per work item: about target_wgs workgroups over all (tile, kv
  // head) pairs, at least one 32-key chunk per wave
  long long split = (total_keys * Hkv + target_wgs - 1) / std::max(1, target_wgs);
  split = std::max<long long>(32 * p.w, (split + 31) / 32 * 32);
  auto parts_for = [&](long long sp) {
    long long n = 0;
    for (const auto& t : tiles) {
      const long long c = (t.kend + sp - 1) / sp;
      if (c > 1) n += c;
    }
    return n;
  };
  while (parts_for(split) > max_parts) split *= 2;
  for (const auto& t : tiles) {
    const int c = static_cast<int>((t.kend + split - 1) / split);
    if (c <= 1) {
      p.items.push_back(AttnItem{t.row0, t.nrows, t.pos0, t.seq, 0, t.kend, -1, 0});
      continue;
    }
    p.groups.push_back(AttnGroup{t.row0, t.nrows, p.n_parts, c});
    for (int i = 0; i < c; ++i) {
      const int t0 = static_cast<int>(i * split);
      const int t1 = static_cast<int>(std::min<long long>(t.kend, (i + 1) * split));
      p.items.push_back(AttnItem{t.row0, t.nrows, t.pos0, t.seq, t0, t1, p.n_parts + i, 0});
    }
    p.n_parts += c;
  }
  // longest key ranges first: workgroups start in this order, so the short
  // items fill in behind the long ones instead of trailing after them
  std::stable_sort(p.items.begin(), p.items.end(),
                   [](const AttnItem& x, const AttnItem& y) { return x.t1 - x.t0 > y.t1 - y.t0; });
  return p;
}

}  // namespace spec
