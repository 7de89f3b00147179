// Host-only part of libooo: error reporting, version and trie packing.
#include <cstdio>
#include <cstring>
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
// are found by walking the parent's child list (first child, next sibling),
// kept in stack arrays bounded by the 1024-node limit of the device kernels
// (the ancestor masks of the attention and accept kernels hold at most 16
// words), so the call keeps no state and allocates nothing.  The ancestor
// bitmask of a node is its parent's mask plus its own bit, which is valid
// because a parent is always created before its children.
constexpr int32_t kMaxTrieNodes = 1024;

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
    OOO_REQUIRE(max_nodes <= kMaxTrieNodes, OOO_ERR_UNSUPPORTED, "max_nodes %d exceeds %d", max_nodes,
                kMaxTrieNodes);
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

    int32_t first_child[kMaxTrieNodes], next_sibling[kMaxTrieNodes];
    first_child[0] = -1;
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
        int32_t ch = first_child[cur];
        while (ch >= 0 && token[ch] != t) ch = next_sibling[ch];
        if (ch >= 0) {
          cur = ch;
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
        first_child[node] = -1;
        next_sibling[node] = first_child[cur];  // newest first; order does not affect the trie
        first_child[cur] = node;
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

// Lanes of one retrieval round (Section 4.4, Suffix matching; Eq. 3).  One
// pass over the bank computes, for every position i, the longest k <=
// max_suffix with bank[i-k, i) equal to the last k committed tokens; the
// suffix length used is the largest k at a position that starts a non-empty
// continuation (not EOS, not the bank end), and every such position with at
// least that match proposes its continuation, in bank order.
extern "C" int ooo_hint_merge(const int32_t* bank, int64_t bank_len, int32_t eos_token, const int32_t* committed,
                              int32_t n_committed, int32_t max_suffix, int32_t max_len,
                              const int32_t* native_tokens, const int32_t* native_offsets, int32_t n_native,
                              int32_t n_lanes, int32_t* out_tokens, int64_t out_cap, int32_t* out_offsets,
                              int32_t* n_out, int32_t* n_hint, int32_t* suffix_len) {
  try {
    OOO_REQUIRE(n_out && n_hint && suffix_len && out_offsets, OOO_ERR_INVALID, "ooo_hint_merge: null output");
    *n_out = 0;
    *n_hint = 0;
    *suffix_len = 0;
    OOO_REQUIRE(bank_len >= 0 && n_committed >= 0 && n_native >= 0 && n_lanes >= 0 && out_cap >= 0,
                OOO_ERR_INVALID, "ooo_hint_merge: negative size");
    OOO_REQUIRE(bank_len == 0 || bank, OOO_ERR_INVALID, "ooo_hint_merge: bank is null");
    OOO_REQUIRE(n_committed == 0 || committed, OOO_ERR_INVALID, "ooo_hint_merge: committed is null");
    OOO_REQUIRE(max_suffix >= 1 && max_len >= 1, OOO_ERR_INVALID,
                "ooo_hint_merge: max_suffix (%d) and max_len (%d) must be >= 1", max_suffix, max_len);
    OOO_REQUIRE(native_offsets, OOO_ERR_INVALID, "ooo_hint_merge: native_offsets is null");
    OOO_REQUIRE(native_offsets[0] == 0, OOO_ERR_INVALID, "ooo_hint_merge: native_offsets[0] must be 0");
    for (int32_t c = 0; c < n_native; ++c)
      OOO_REQUIRE(native_offsets[c + 1] >= native_offsets[c], OOO_ERR_INVALID,
                  "ooo_hint_merge: native_offsets must be non-decreasing (at %d)", c);
    OOO_REQUIRE(native_offsets[n_native] == 0 || native_tokens, OOO_ERR_INVALID,
                "ooo_hint_merge: native_tokens is null");
    for (int32_t t = 0; t < native_offsets[n_native]; ++t)
      OOO_REQUIRE(native_tokens[t] >= 0, OOO_ERR_INVALID, "ooo_hint_merge: negative native token at %d", t);
    OOO_REQUIRE(n_lanes == 0 || out_cap == 0 || out_tokens, OOO_ERR_INVALID, "ooo_hint_merge: out_tokens is null");

    const int32_t K = max_suffix < n_committed ? max_suffix : n_committed;
    const int32_t* tail = committed + n_committed;  // tail[-k] is the k-th last committed token
    auto match_before = [&](int64_t i) {           // longest k with bank[i-k, i) == last k committed
      int32_t k = 0;
      while (k < K && i - k - 1 >= 0 && bank[i - k - 1] == tail[-k - 1]) ++k;
      return k;
    };
    auto starts_proposal = [&](int64_t i) { return i < bank_len && bank[i] != eos_token; };
    int32_t best = 0;
    if (K > 0)
      for (int64_t i = 1; i < bank_len && best < K; ++i)
        if (starts_proposal(i)) {
          const int32_t k = match_before(i);
          if (k > best) best = k;
        }

    std::vector<std::vector<int32_t>> lanes;
    if (best > 0)
      for (int64_t i = best; i < bank_len && (int32_t)lanes.size() < n_lanes; ++i) {
        if (!starts_proposal(i) || match_before(i) < best) continue;
        std::vector<int32_t> cont;
        for (int64_t j = i; j < bank_len && bank[j] != eos_token && (int32_t)cont.size() < max_len; ++j)
          cont.push_back(bank[j]);
        bool seen = false;
        for (const auto& l : lanes) seen = seen || l == cont;
        if (!seen) lanes.push_back(std::move(cont));
      }
    const int32_t hints = (int32_t)lanes.size();
    for (int32_t c = 0; c < n_native && (int32_t)lanes.size() < n_lanes; ++c)
      lanes.emplace_back(native_tokens + native_offsets[c], native_tokens + native_offsets[c + 1]);

    int64_t total = 0;
    for (const auto& l : lanes) total += (int64_t)l.size();
    OOO_REQUIRE(total <= out_cap, OOO_ERR_CAPACITY, "ooo_hint_merge: %lld merged tokens exceed out_cap %lld",
                (long long)total, (long long)out_cap);
    int64_t pos = 0;
    out_offsets[0] = 0;
    for (size_t c = 0; c < lanes.size(); ++c) {
      for (int32_t t : lanes[c]) out_tokens[pos++] = t;
      out_offsets[c + 1] = (int32_t)pos;
    }
    *n_out = (int32_t)lanes.size();
    *n_hint = hints;
    *suffix_len = best;
    return ooo::ok();
  } catch (...) {
    return ooo::fail(OOO_ERR_INVALID, "ooo_hint_merge: internal error");
  }
}
