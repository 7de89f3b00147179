// Host-only part of libooo: error reporting, version and trie packing.
#include <cstdio>
#include <cstring>
#include <unordered_map>
#include <vector>

#include "ooo_internal.h"

namespace ooo {

static thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_err[0] = '\0';
  return OOO_OK;
}

}  // namespace ooo

extern "C" const char* ooo_last_error(void) { return ooo::g_err; }

extern "C" int ooo_version(void) { return OOO_ABI_VERSION; }

// Candidate trie (Section 3, ToolSpec loop; Section 4.4, fixed candidate
// budget with hint lanes first; Section 4.5, one candidate tree).  Children
// are found through a hash map keyed by (parent, token); the ancestor bitmask
// of a node is its parent's mask plus its own bit, which is valid because a
// parent is always created before its children.
extern "C" int ooo_pack_tree(int32_t root_token, const int32_t* cand_tokens,
                             const int32_t* cand_offsets, int32_t n_cand, int32_t max_nodes,
                             int32_t max_depth, int32_t* token, int32_t* parent, int32_t* depth,
                             uint64_t* anc_mask, int32_t mask_words, int32_t* n_nodes,
                             int32_t* n_truncated) {
  try {
    OOO_REQUIRE(n_cand >= 0, OOO_ERR_INVALID, "n_cand must be >= 0 (got %d)", n_cand);
    OOO_REQUIRE(cand_offsets != nullptr, OOO_ERR_INVALID, "cand_offsets is null");
    OOO_REQUIRE(token && parent && depth && anc_mask && n_nodes && n_truncated, OOO_ERR_INVALID,
                "an output pointer is null");
    OOO_REQUIRE(max_nodes >= 1, OOO_ERR_INVALID, "max_nodes must be >= 1 (got %d)", max_nodes);
    OOO_REQUIRE(max_depth >= 0, OOO_ERR_INVALID, "max_depth must be >= 0 (got %d)", max_depth);
    OOO_REQUIRE(mask_words >= 1 && (int64_t)mask_words * 64 >= max_nodes, OOO_ERR_INVALID,
                "mask_words=%d cannot hold %d nodes", mask_words, max_nodes);
    OOO_REQUIRE(root_token >= 0, OOO_ERR_INVALID, "root_token must be >= 0");
    OOO_REQUIRE(cand_offsets[0] == 0, OOO_ERR_INVALID, "cand_offsets[0] must be 0");
    for (int32_t c = 0; c < n_cand; ++c)
      OOO_REQUIRE(cand_offsets[c + 1] >= cand_offsets[c], OOO_ERR_INVALID,
                  "cand_offsets must be non-decreasing (at %d)", c);
    const int32_t total = cand_offsets[n_cand];
    OOO_REQUIRE(total == 0 || cand_tokens != nullptr, OOO_ERR_INVALID, "cand_tokens is null");
    for (int32_t t = 0; t < total; ++t)
      OOO_REQUIRE(cand_tokens[t] >= 0, OOO_ERR_INVALID, "negative token at position %d", t);

    std::unordered_map<uint64_t, int32_t> child;  // (parent << 32 | token) -> node
    child.reserve(2 * (size_t)max_nodes);
    int32_t n = 1;
    int32_t dropped = 0;
    token[0] = root_token;
    parent[0] = -1;
    depth[0] = 0;
    std::memset(anc_mask, 0, sizeof(uint64_t) * (size_t)max_nodes * mask_words);
    anc_mask[0] = 1ull;
    for (int32_t c = 0; c < n_cand; ++c) {
      const int32_t a = cand_offsets[c], b = cand_offsets[c + 1];
      int32_t cur = 0;
      for (int32_t pos = 0; pos < b - a; ++pos) {
        if (pos >= max_depth) {
          dropped += (b - a) - pos;
          break;
        }
        const int32_t t = cand_tokens[a + pos];
        const uint64_t key = ((uint64_t)(uint32_t)cur << 32) | (uint32_t)t;
        auto it = child.find(key);
        if (it != child.end()) {
          cur = it->second;
          continue;
        }
        if (n >= max_nodes) {
          dropped += (b - a) - pos;
          break;
        }
        const int32_t node = n++;
        token[node] = t;
        parent[node] = cur;
        depth[node] = depth[cur] + 1;
        uint64_t* row = anc_mask + (size_t)node * mask_words;
        const uint64_t* prow = anc_mask + (size_t)cur * mask_words;
        for (int32_t w = 0; w < mask_words; ++w) row[w] = prow[w];
        row[node >> 6] |= 1ull << (node & 63);
        child.emplace(key, node);
        cur = node;
      }
    }
    *n_nodes = n;
    *n_truncated = dropped;
    return ooo::ok();
  } catch (...) {
    return ooo::fail(OOO_ERR_INVALID, "ooo_pack_tree: internal error");
  }
}
