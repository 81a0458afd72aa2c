// Test driver for the library's host page allocator (pure C++): reads a script
// of operations on stdin and prints every page table after each step.
//   "E seq length"  ensure   |  "T seq length"  truncate
#include <cstdio>
#include <map>
#include <vector>

#include "pages.h"

int main() {
  int num_pages = 0;
  if (std::scanf("%d", &num_pages) != 1) return 2;
  spec::PagePool pool(num_pages, 16);
  std::map<long long, std::vector<int32_t>> tabs;
  char op;
  long long seq, len;
  while (std::scanf(" %c %lld %lld", &op, &seq, &len) == 3) {
    auto& t = tabs[seq];
    if (op == 'E') {
      const bool ok = pool.ensure(t, len);
      std::printf("%s", ok ? "ok" : "oom");
    } else {
      pool.truncate(t, len);
      std::printf("ok");
    }
    for (auto& kv : tabs) {
      std::printf(" |%lld:", kv.first);
      for (int32_t p : kv.second) std::printf(" %d", p);
    }
    std::printf("\n");
  }
  return 0;
}
