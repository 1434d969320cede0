// Window-safe prefix cache tree (host).
//
// "SWA-Aware Prefix Cache Tree": a radix tree over token ids whose nodes carry,
// per token, the FULL attention KV slot and the SWA KV slot (dual indices).
// Equal tokens no longer imply reusable KV: the SWA slots of a cached prefix
// may have been released. A match is therefore clipped to the longest prefix
// length P whose window is intact, i.e. the W - 1 tokens before P (the keys
// the first new query at position P reads from the SWA pool) all hold valid
// SWA slots; anything beyond is a miss. SWA slots outside the window can be
// released on their own while the FULL slots stay (the prefix stays usable by
// FULL layers), or whole segments can be evicted.
//
// Nodes hold a run of tokens (path compression); children are keyed by their
// first token.
#include <stdint.h>

#include <map>
#include <memory>
#include <new>
#include <vector>

#include "hswa.h"

namespace {

struct Node {
  std::vector<int32_t> tok;
  std::vector<int64_t> full, swa;  // per token: slot or -1
  std::map<int32_t, std::unique_ptr<Node>> kids;

  Node() = default;
  Node(const Node &) = delete;
  Node &operator=(const Node &) = delete;
  // A path may hold any number of branch points: descendants are detached
  // onto a work list and freed one by one, so that freeing a subtree (at
  // teardown, eviction or a cut) never recurses once per level.
  ~Node() {
    std::vector<std::unique_ptr<Node>> pending;
    for (auto &kv : kids) pending.push_back(std::move(kv.second));
    kids.clear();
    while (!pending.empty()) {
      std::unique_ptr<Node> n = std::move(pending.back());
      pending.pop_back();
      for (auto &kv : n->kids) pending.push_back(std::move(kv.second));
      n->kids.clear();
    }
  }

  // Splits this node after its first `at` tokens; the tail becomes the only child.
  void split(size_t at) {
    auto tail = std::make_unique<Node>();
    tail->tok.assign(tok.begin() + at, tok.end());
    tail->full.assign(full.begin() + at, full.end());
    tail->swa.assign(swa.begin() + at, swa.end());
    tail->kids.swap(kids);
    tok.resize(at);
    full.resize(at);
    swa.resize(at);
    const int32_t key = tail->tok[0];
    kids.emplace(key, std::move(tail));
  }
};

// Tokens, SWA-valid tokens and nodes of the subtree at n (n included), by an
// explicit work list: no recursion, whatever the depth.
struct SubtreeCount {
  int64_t tokens = 0, swa_valid = 0, nodes = 0;
};

SubtreeCount count_subtree(const Node &n) {
  SubtreeCount c;
  std::vector<const Node *> todo{&n};
  while (!todo.empty()) {
    const Node *x = todo.back();
    todo.pop_back();
    ++c.nodes;
    c.tokens += (int64_t)x->tok.size();
    for (int64_t s : x->swa) c.swa_valid += s >= 0;
    for (const auto &kv : x->kids) todo.push_back(kv.second.get());
  }
  return c;
}

}  // namespace

struct hswa_prefix_tree {
  int32_t window = 1;
  Node root;  // holds no tokens
};

extern "C" {

hswa_status hswa_prefix_tree_create(int32_t window, hswa_prefix_tree **out) {
  if (!out || window < 1) return HSWA_ERR_INVALID_ARG;
  *out = nullptr;
  hswa_prefix_tree *t = new (std::nothrow) hswa_prefix_tree();
  if (!t) return HSWA_ERR_CAPACITY;
  t->window = window;
  *out = t;
  return HSWA_OK;
}

void hswa_prefix_tree_destroy(hswa_prefix_tree *t) { delete t; }

hswa_status hswa_prefix_tree_insert(hswa_prefix_tree *t, const int32_t *tokens, int64_t n, const int64_t *full_slots,
                                    const int64_t *swa_slots) {
  if (!t || n < 0 || (n > 0 && (!tokens || !full_slots || !swa_slots))) return HSWA_ERR_INVALID_ARG;
  try {
    Node *node = &t->root;
    int64_t i = 0;
    while (i < n) {
      auto it = node->kids.find(tokens[i]);
      if (it == node->kids.end()) {  // a new leaf holds the rest
        auto leaf = std::make_unique<Node>();
        leaf->tok.assign(tokens + i, tokens + n);
        leaf->full.assign(full_slots + i, full_slots + n);
        leaf->swa.assign(swa_slots + i, swa_slots + n);
        node->kids.emplace(tokens[i], std::move(leaf));
        return HSWA_OK;
      }
      Node *c = it->second.get();
      size_t k = 0;
      while (k < c->tok.size() && i + (int64_t)k < n && c->tok[k] == tokens[i + k]) ++k;
      if (k < c->tok.size()) c->split(k);
      for (size_t j = 0; j < k; ++j) {  // newer slots replace older ones
        c->full[j] = full_slots[i + j];
        c->swa[j] = swa_slots[i + j];
      }
      i += (int64_t)k;
      node = c;
    }
  } catch (...) {
    return HSWA_ERR_CAPACITY;
  }
  return HSWA_OK;
}

hswa_status hswa_prefix_tree_match(const hswa_prefix_tree *t, const int32_t *tokens, int64_t n, int64_t *full_len,
                                   int64_t *safe_len, int64_t *full_slots_out, int64_t *swa_slots_out) {
  if (!t || n < 0 || (n > 0 && !tokens)) return HSWA_ERR_INVALID_ARG;
  // Walk while tokens are equal and the FULL slot is held.
  int64_t len = 0;
  int64_t last_bad_swa = -1;  // last matched position without an SWA slot
  std::vector<int64_t> bad_before;  // bad_before[p] = last invalid SWA position < p
  try {
    bad_before.reserve((size_t)n + 1);
    bad_before.push_back(-1);
    const Node *node = &t->root;
    bool go = true;
    while (go && len < n) {
      auto it = node->kids.find(tokens[len]);
      if (it == node->kids.end()) break;
      const Node *c = it->second.get();
      size_t k = 0;
      for (; k < c->tok.size() && len < n; ++k) {
        if (c->tok[k] != tokens[len] || c->full[k] < 0) {
          go = false;
          break;
        }
        if (full_slots_out) full_slots_out[len] = c->full[k];
        if (swa_slots_out) swa_slots_out[len] = c->swa[k];
        if (c->swa[k] < 0) last_bad_swa = len;
        ++len;
        bad_before.push_back(last_bad_swa);
      }
      if (k < c->tok.size()) break;
      node = c;
    }
  } catch (...) {
    return HSWA_ERR_CAPACITY;
  }
  // Largest P <= len whose window keys [max(0, P - W + 1), P) all hold SWA slots.
  int64_t safe = 0;
  for (int64_t p = len; p > 0; --p) {
    const int64_t lo = p - t->window + 1 > 0 ? p - t->window + 1 : 0;
    if (bad_before[p] < lo) {
      safe = p;
      break;
    }
  }
  if (full_len) *full_len = len;
  if (safe_len) *safe_len = safe;
  return HSWA_OK;
}

hswa_status hswa_prefix_tree_release_swa(hswa_prefix_tree *t, const int32_t *tokens, int64_t n, int64_t upto,
                                         int64_t *released) {
  if (!t || n < 0 || upto < 0 || (n > 0 && !tokens)) return HSWA_ERR_INVALID_ARG;
  int64_t cnt = 0, pos = 0;
  Node *node = &t->root;
  while (pos < n && pos < upto) {
    auto it = node->kids.find(tokens[pos]);
    if (it == node->kids.end()) break;
    Node *c = it->second.get();
    size_t k = 0;
    for (; k < c->tok.size() && pos < n && pos < upto && c->tok[k] == tokens[pos]; ++k, ++pos) {
      if (c->swa[k] >= 0) {
        c->swa[k] = -1;
        ++cnt;
      }
    }
    if (k < c->tok.size()) break;
    node = c;
  }
  if (released) *released = cnt;
  return HSWA_OK;
}

hswa_status hswa_prefix_tree_evict(hswa_prefix_tree *t, const int32_t *tokens, int64_t n, int64_t keep,
                                   int64_t *evicted) {
  if (!t || n < 0 || keep < 0 || (n > 0 && !tokens)) return HSWA_ERR_INVALID_ARG;
  int64_t cnt = 0;
  if (keep >= n) {
    if (evicted) *evicted = 0;
    return HSWA_OK;
  }
  // Find the node holding position `keep` on this path and cut there.
  Node *node = &t->root;
  int64_t pos = 0;
  try {
    while (true) {
      auto it = node->kids.find(tokens[pos]);
      if (it == node->kids.end()) break;  // nothing cached at or beyond keep on this path
      Node *c = it->second.get();
      size_t k = 0;
      while (k < c->tok.size() && pos + (int64_t)k < n && c->tok[k] == tokens[pos + k] && pos + (int64_t)k < keep) ++k;
      if (pos + (int64_t)k == keep) {
        if (k == 0) {  // the whole child subtree goes
          cnt = count_subtree(*c).tokens;
          node->kids.erase(it);
        } else if (k < c->tok.size()) {  // cut inside the node: drop its tail and all children
          if (c->tok[k] == tokens[pos + k]) {
            c->split(k);
            cnt = count_subtree(*c->kids.begin()->second).tokens;
            c->kids.clear();
          }
        } else {  // keep ends exactly after this node: drop the child that continues the path
          auto it2 = c->kids.find(tokens[keep]);
          if (it2 != c->kids.end()) {
            cnt = count_subtree(*it2->second).tokens;
            c->kids.erase(it2);
          }
        }
        break;
      }
      if (k < c->tok.size()) break;  // the path diverges before keep
      pos += (int64_t)k;
      node = c;
    }
  } catch (...) {  // the count's work list could not grow (a split before it keeps the tree valid)
    return HSWA_ERR_CAPACITY;
  }
  if (evicted) *evicted = cnt;
  return HSWA_OK;
}

hswa_status hswa_prefix_tree_stats(const hswa_prefix_tree *t, int64_t *nodes, int64_t *tokens,
                                   int64_t *swa_valid_tokens) {
  if (!t) return HSWA_ERR_INVALID_ARG;
  SubtreeCount c;
  try {
    c = count_subtree(t->root);
  } catch (...) {
    return HSWA_ERR_CAPACITY;
  }
  if (nodes) *nodes = c.nodes - 1;  // the root holds no tokens
  if (tokens) *tokens = c.tokens;
  if (swa_valid_tokens) *swa_valid_tokens = c.swa_valid;
  return HSWA_OK;
}

}  // extern "C"
