// Greedy acceptance and cache compaction (Section 4.5, Verify and commit:
// draft tokens are kept while they match the target's greedy token at their
// parent, the first mismatch ends the run and the target's own token follows;
// only the accepted states are committed to the KV cache).
//
// ooo_accept runs in one block.  Node i "matches" when it is the root or its
// token equals the greedy token of its parent; the match bits of 64 nodes are
// one wavefront ballot, so they land directly in the layout of the ancestor
// bitmask.  A node is accepted iff every ancestor-or-self matches, i.e.
// (anc_mask[i] & ~match) == 0.  Because siblings carry distinct tokens the
// accepted nodes form one root path; its length is a max-reduction over their
// depths and path[depth[i]] = i places each of them.
//
// ooo_kv_compact moves row P + path[d] to row P + d for every layer, KV head,
// K and V.  One block per (layer, head, K|V) slice; each pass reads up to 64
// source rows into registers, synchronises, then writes them.  This is safe
// in place: path is strictly increasing with path[d] >= d, so a pass only
// overwrites rows below every source row of the later passes.
#include "device_common.h"
#include "ooo_internal.h"

namespace ooo {
namespace {

constexpr int kMaxMaskWords = 16;

// All inputs are read once, with every load issued up front (one round trip
// to memory); the parent's greedy token and the bonus are then looked up in
// LDS.  Depths of accepted nodes are below n_nodes <= 1024, so path entries
// from 1024 on are always -1.
constexpr int kMaxNodes = 64 * kMaxMaskWords;
__global__ __launch_bounds__(1024) void accept_kernel(const int32_t* __restrict__ token,
                                                      const int32_t* __restrict__ parent,
                                                      const int32_t* __restrict__ depth,
                                                      const uint64_t* __restrict__ anc, int W,
                                                      const int32_t* __restrict__ ids, int N, int path_cap,
                                                      int32_t* __restrict__ path, int32_t* __restrict__ accept_len,
                                                      int32_t* __restrict__ bonus) {
  __shared__ uint64_t match[kMaxMaskWords];
  __shared__ int32_t ids_s[kMaxNodes];
  __shared__ int32_t path_s[kMaxNodes];
  __shared__ int best_depth;
  const int tid = threadIdx.x;
  const int i = tid;  // one thread per node (blockDim = 64 * W >= N)
  int tk = 0, pa = 0, dp = 0;
  uint64_t am[kMaxMaskWords];
  if (i < N) {
    tk = token[i];
    pa = parent[i];
    dp = depth[i];
    ids_s[i] = ids[i];
#pragma unroll
    for (int w = 0; w < kMaxMaskWords; ++w)
      if (w < W) am[w] = anc[(size_t)i * W + w];
  }
  for (int k = tid; k < kMaxNodes; k += blockDim.x) path_s[k] = -1;
  if (tid == 0) best_depth = 0;
  __syncthreads();
  // match bits, one ballot per 64 nodes
  const bool m = i < N && (i == 0 || (pa >= 0 && pa < N && tk == ids_s[pa]));
  const uint64_t bits = __ballot(m);
  if ((tid & 63) == 0 && tid < 64 * W) match[tid >> 6] = bits;
  __syncthreads();
  if (i < N) {
    bool ok = true;
#pragma unroll
    for (int w = 0; w < kMaxMaskWords; ++w)
      if (w < W) ok = ok && ((am[w] & ~match[w]) == 0);
    if (ok) {
      if (dp < path_cap && dp < kMaxNodes) path_s[dp] = i;
      atomicMax(&best_depth, dp);
    }
  }
  __syncthreads();
  // An accepted node deeper than path[] holds (a trie deeper than the
  // caller's max_depth) is reported as accept_len = -1 with an empty path:
  // the step commits nothing rather than a shortened path.
  const bool overflow = best_depth >= path_cap || best_depth >= kMaxNodes;
  for (int k = tid; k < path_cap; k += blockDim.x) path[k] = (!overflow && k < kMaxNodes) ? path_s[k] : -1;
  if (tid == 0) {
    const int L = best_depth;
    *accept_len = overflow ? -1 : L;
    *bonus = overflow ? -1 : ids_s[path_s[L]];
  }
}

__global__ __launch_bounds__(256) void kv_compact_kernel(uint8_t* __restrict__ k, uint8_t* __restrict__ v,
                                                         int Hkv, long long cap, int row_bytes, int P,
                                                         const int32_t* __restrict__ P_dev, int N,
                                                         const int32_t* __restrict__ path,
                                                         const int32_t* __restrict__ accept_len, int path_cap) {
  const int slice = blockIdx.x;  // (layer * Hkv + head) * 2 + (K or V)
  uint8_t* base = ((slice & 1) ? v : k) + (size_t)(slice >> 1) * cap * row_bytes;
  const int chunks = row_bytes / 16;  // 16-byte pieces per row
  constexpr int R = 4;                // pieces per thread per pass
  const int rows_per_pass = (256 * R) / chunks;
  // The first pass's path entries are read together with the accepted
  // length (one round trip instead of two); entries past it go unused.
  int first_src[R];
#pragma unroll
  for (int i = 0; i < R; ++i) {
    const int item = threadIdx.x + 256 * i;
    const int d = 1 + item / chunks;
    first_src[i] = (item < rows_per_pass * chunks && d < path_cap && d < N) ? path[d] : -1;
  }
  int L = *accept_len;  // -1 (overflow reported by ooo_accept): nothing to move
  if (L > path_cap - 1) L = path_cap - 1;
  if (P_dev) P = min(max(*P_dev, 0), P);  // device prefix, bounded by the launch value
  for (int d0 = 1; d0 <= L; d0 += rows_per_pass) {
    u32x4 buf[R];
    int dst[R];
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int item = threadIdx.x + 256 * i;
      const int d = d0 + item / chunks, ch = item % chunks;
      dst[i] = -1;
      if (item < rows_per_pass * chunks && d <= L && d < N) {
        const int src = d0 == 1 ? first_src[i] : path[d];
        if (src >= 0 && src < N) {
          buf[i] = ld16(base + (size_t)(P + src) * row_bytes + 16 * ch);
          dst[i] = d;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < R; ++i) {
      const int item = threadIdx.x + 256 * i;
      if (dst[i] >= 0) st16(base + (size_t)(P + dst[i]) * row_bytes + 16 * (item % chunks), buf[i]);
    }
    __syncthreads();
  }
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" int ooo_accept(const int32_t* token, const int32_t* parent, const int32_t* depth,
                          const uint64_t* anc_mask, int32_t mask_words, const int32_t* argmax_ids,
                          int32_t n_nodes, int32_t max_depth, int32_t path_cap, int32_t* path,
                          int32_t* accept_len, int32_t* bonus_token, void* stream) {
  OOO_REQUIRE(token && parent && depth && anc_mask && argmax_ids && path && accept_len && bonus_token,
              OOO_ERR_INVALID, "ooo_accept: null pointer");
  OOO_REQUIRE(n_nodes >= 1, OOO_ERR_INVALID, "ooo_accept: n_nodes must be >= 1");
  OOO_REQUIRE(max_depth >= 0 && path_cap >= 1, OOO_ERR_INVALID,
              "ooo_accept: max_depth (%d) must be >= 0 and path_cap (%d) >= 1", max_depth, path_cap);
  OOO_REQUIRE(path_cap >= max_depth + 1, OOO_ERR_CAPACITY,
              "ooo_accept: path of %d entries cannot hold a root path of depth %d", path_cap, max_depth);
  OOO_REQUIRE(mask_words >= 1 && mask_words <= kMaxMaskWords && (int64_t)mask_words * 64 >= n_nodes,
              OOO_ERR_INVALID, "ooo_accept: mask_words=%d cannot describe %d nodes (max %d words)", mask_words,
              n_nodes, kMaxMaskWords);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  int threads = 64 * mask_words;
  if (threads > 1024) threads = 1024;
  accept_kernel<<<1, threads, 0, st>>>(token, parent, depth, anc_mask, mask_words, argmax_ids, n_nodes, path_cap,
                                       path, accept_len, bonus_token);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_accept: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_kv_compact(void* k_cache, void* v_cache, int32_t n_layers, int32_t n_kv_heads, int64_t cap,
                              int32_t head_dim, ooo_dtype dt, int32_t prefix_len, const int32_t* prefix_len_dev,
                              int32_t n_nodes,
                              const int32_t* path, const int32_t* accept_len, int32_t path_cap, void* stream) {
  OOO_REQUIRE(k_cache && v_cache && path && accept_len, OOO_ERR_INVALID, "ooo_kv_compact: null pointer");
  OOO_REQUIRE(n_layers >= 1 && n_kv_heads >= 1 && head_dim >= 1 && n_nodes >= 1 && path_cap >= 1,
              OOO_ERR_INVALID, "ooo_kv_compact: sizes must be positive");
  OOO_REQUIRE(prefix_len >= 0 && (int64_t)prefix_len + n_nodes <= cap, OOO_ERR_INVALID,
              "ooo_kv_compact: prefix_len + n_nodes (%lld) exceeds cap (%lld)", (long long)prefix_len + n_nodes,
              (long long)cap);
  OOO_REQUIRE(dt == OOO_F32 || dt == OOO_BF16, OOO_ERR_INVALID, "ooo_kv_compact: unknown dtype %d", (int)dt);
  const int esz = dt == OOO_F32 ? 4 : 2;
  const int row_bytes = head_dim * esz;
  OOO_REQUIRE(row_bytes % 16 == 0 && row_bytes <= 1024 * 16, OOO_ERR_UNSUPPORTED,
              "ooo_kv_compact: row of %d bytes is not a multiple of 16 (or too long)", row_bytes);
  OOO_REQUIRE((int64_t)n_layers * n_kv_heads * 2 <= 0x7FFFFFFF, OOO_ERR_UNSUPPORTED, "ooo_kv_compact: too many slices");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid(n_layers * n_kv_heads * 2);
  if (esz == 2)
    kv_compact_kernel<<<grid, 256, 0, st>>>((uint8_t*)k_cache, (uint8_t*)v_cache, n_kv_heads, cap, row_bytes,
                                                prefix_len, prefix_len_dev, n_nodes, path, accept_len, path_cap);
  else
    kv_compact_kernel<<<grid, 256, 0, st>>>((uint8_t*)k_cache, (uint8_t*)v_cache, n_kv_heads, cap, row_bytes,
                                                prefix_len, prefix_len_dev, n_nodes, path, accept_len, path_cap);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_kv_compact: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
