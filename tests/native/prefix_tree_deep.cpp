// A prefix tree whose one path holds N branch points (N levels), built
// directly on the tree's nodes (through the API it would take N inserts of
// growing prefixes): counting it, matching along it, evicting a deep subtree
// and tearing it down must not recurse once per level. Run with a small stack.
#include <cstdio>
#include <cstdlib>
#include <numeric>

#include "../../paper_2607_13095_amd/csrc/prefix_tree.cpp"

#define CHECK(c)                                        \
  do {                                                  \
    if (!(c)) {                                         \
      std::fprintf(stderr, "check failed: %s\n", #c);   \
      return 1;                                         \
    }                                                   \
  } while (0)

int main(int argc, char **argv) {
  const int n = argc > 1 ? std::atoi(argv[1]) : 200000;
  hswa_prefix_tree *t = nullptr;
  CHECK(hswa_prefix_tree_create(16, &t) == HSWA_OK);
  // path node i holds token i; node i - 1 (the root for i = 0) also has a
  // one-token side leaf -1 - i, so every level is a branch point
  Node *node = &t->root;
  for (int i = 0; i < n; ++i) {
    auto side = std::make_unique<Node>();
    side->tok = {-1 - i};
    side->full = {i};
    side->swa = {-1};
    node->kids.emplace(-1 - i, std::move(side));
    auto next = std::make_unique<Node>();
    next->tok = {i};
    next->full = {i};
    next->swa = {i};
    Node *raw = next.get();
    node->kids.emplace(i, std::move(next));
    node = raw;
  }
  int64_t nodes = 0, tokens = 0, swa_valid = 0;
  CHECK(hswa_prefix_tree_stats(t, &nodes, &tokens, &swa_valid) == HSWA_OK);
  CHECK(nodes == 2 * (int64_t)n && tokens == 2 * (int64_t)n && swa_valid == n);

  std::vector<int32_t> path(n);
  std::iota(path.begin(), path.end(), 0);
  int64_t full_len = 0, safe_len = 0;
  CHECK(hswa_prefix_tree_match(t, path.data(), n, &full_len, &safe_len, nullptr, nullptr) == HSWA_OK);
  CHECK(full_len == n && safe_len == n);

  // cut after position k: path nodes k .. n-1 and the side leaves below node k go
  const int k = n / 2;
  int64_t evicted = 0;
  CHECK(hswa_prefix_tree_evict(t, path.data(), n, k, &evicted) == HSWA_OK);
  CHECK(evicted == 2 * (int64_t)(n - k) - 1);
  CHECK(hswa_prefix_tree_stats(t, &nodes, &tokens, &swa_valid) == HSWA_OK);
  CHECK(nodes == 2 * (int64_t)k + 1 && tokens == nodes);

  hswa_prefix_tree_destroy(t);  // k levels left
  std::printf("ok %d\n", n);
  return 0;
}
