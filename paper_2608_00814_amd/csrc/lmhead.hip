// LM head and greedy token of every trie node (Eq. 1: the next committed
// token is the target's most likely one; ties go to the lowest index).
//
// bf16 path: the product is W[V][H] x X[N][H]^T, a skinny GEMM that streams
// W from HBM once; it is bound by HBM bandwidth, so the design is about
// keeping enough whole cache lines in flight:
//  * A persistent grid (one block per CU) walks 128-row vocabulary tiles
//    round-robin; the K dimension is cut into 64-element chunks.  The last,
//    partial round of tiles is dealt out in 32-row groups (one per compute
//    wave), so that no block streams more than one group beyond the average
//    (1187 tiles on 256 blocks: 4 tiles + 2 or 3 groups each, instead of 4
//    or 5 tiles).
//  * The streaming core (stream_core.h): two loader waves copy each W
//    chunk (128 rows x 128 B) and a third the X chunk (all nodes x 128 B)
//    straight into an LDS ring with global_load_lds; four compute waves own
//    32 rows each and run the MFMAs from LDS, never issuing global loads in
//    the loop.
//  * Each lane ends a tile with 16 logits of one node; the per-node argmax is
//    kept in registers across tiles, merged across the block's waves in LDS
//    and across blocks by a small finalize kernel (value, then lowest index).
#include <math.h>

#include "device_common.h"
#include "ooo_internal.h"
#include "stream_core.h"

namespace ooo {
namespace {

struct Cand {
  float v;
  int i;
};

constexpr int kLmRows = kStreamRows;  // vocabulary rows per tile (4 waves x 32)

template <int NB, bool PACKED>
__global__ __launch_bounds__(kStreamThreads) void lmhead_bf16_kernel(const uint16_t* __restrict__ X,
                                                          const uint16_t* __restrict__ Wt, int N, int H, int V,
                                                          Cand* __restrict__ partial, float* __restrict__ logits) {
  using R = StreamRing<NB>;
  static_assert(R::BYTES + 4 * 32 * NB * sizeof(Cand) <= 160 * 1024, "LDS capacity");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[R::BYTES];
  __shared__ Cand red[4][32 * NB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int chunks = H / 64;
  const int b = (int)blockIdx.x, grid = (int)gridDim.x;
  const int ntiles_all = (V + kLmRows - 1) / kLmRows;
  const int full_rounds = ntiles_all / grid;                  // rounds of whole tiles for every block
  const int rem_groups = (ntiles_all - full_rounds * grid) * 4;  // 32-row groups of the last round
  const int my_tiles = full_rounds + (rem_groups > b ? 1 : 0);
  const int total = my_tiles * chunks;  // chunks this block streams
  // 32-row group of slot s (compute wave s) in the block's tile t, or -1
  auto group_of = [&](int t, int s) {
    if (t < full_rounds) return 4 * (b + t * grid) + s;
    const int rg = b + s * grid;
    return rg < rem_groups ? 4 * full_rounds * grid + rg : -1;
  };

  if (wave >= 4) {
    // -------------------------------------- loaders: W slots 0-1 (4), 2-3 (5), X (6)
    const bool is_x = wave == 6;
    const int s_lo = 2 * (wave - 4);  // first W slot of this loader
    // Per-slot source of the tile whose chunks are being issued, set once
    // per tile: the group's first chunk and the element step per chunk.  An
    // empty slot (last round only) copies a line of X instead (step 0),
    // which sits in L2, so that every chunk is the same number of DMA
    // instructions.
    int issue_tile = -1;
    const uint16_t* sbase[4];
    int sstep[4];
    auto set_tile = [&](int t) {
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) {
        const int gi = group_of(t, s4);
        if (gi < 0) {
          sbase[s4] = X + (size_t)(b % N) * H + min(lane * 8, H - 8);
          sstep[s4] = 0;
        } else if (PACKED) {
          // the group's chunk is a contiguous 4 KiB run of the tile's 16 KiB
          // block, already swizzled
          sbase[s4] = Wt + ((size_t)(gi / 4) * chunks * kLmRows + 32 * (gi % 4)) * 64 + lane * 8;
          sstep[s4] = kLmRows * 64;
        } else {
          sbase[s4] = Wt + (size_t)32 * gi * H;  // group row 0; rows and pieces per lane below
          sstep[s4] = 64;
        }
      }
      issue_tile = t;
    };
    auto issue = [&](int q, int stage) {
      const int t = q / chunks;
      const int kc = q % chunks;
      if (!is_x) {
        uint8_t* dst = lds + stage * R::WS;
        if (t != issue_tile) set_tile(t);
        // slot s4's 32 rows go to LDS rows 32 s4 .. 32 s4 + 31 of the stage
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
          if (s4 / 2 != s_lo / 2) continue;
          if (PACKED || sstep[s4] == 0) {
            dma_w_slot_packed(sbase[s4] + kc * sstep[s4], sstep[s4], dst + s4 * 4096);
          } else {
            dma_w_slot_rows(Wt, H, 32 * group_of(t, s4), V, kc, dst + s4 * 4096, lane);
          }
        }
      } else {
        dma_x_chunk<NB>(X, N, H, kc, lds + R::XREG + stage * R::XS, lane);
      }
    };
    if (is_x) loader_stream<R::NS, R::XDMA>(total, issue);
    else loader_stream<R::NS, R::WDMA>(total, issue);
    __syncthreads();  // matches the compute waves' final reduction barrier
    return;
  }

  // ------------------------------------------------------------------ compute
  const int c = lane & 31, u = lane >> 5;
  uint32_t off[4];
  frag_offsets(lane, off);
  const uint32_t wrow = wave * 32 * 128;

  float bestv[NB];
  int besti[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    bestv[nb] = -INFINITY;
    besti[nb] = 0x7FFFFFFF;
  }
  f32x16 acc[NB];
  int gi = -1;  // this wave's 32-row group in the current tile
  for (int q = 0; q < total; ++q) {
    const int kc = q % chunks;
    if (kc == 0) {
      gi = group_of(q / chunks, wave);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x16{};
    }
    const int stage = q % R::NS;
    wg_barrier();
    if (gi < 0) continue;  // empty slot of the last round (barriers only)
    chunk_mfma<NB>(lds + stage * R::WS + wrow, lds + R::XREG + stage * R::XS, off, acc);

    if (kc == chunks - 1) {
      // tile done: acc[nb][j] = logit of vocabulary row v0 + 8(j/4) + 4u + j%4, node 32nb + c
      const int v0 = 32 * gi;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int r = v0 + 8 * (j / 4) + 4 * u + (j % 4);
          if (r < V && acc[nb][j] > bv) {
            bv = acc[nb][j];
            bi = r;
          }
        }
        const float ov = shfl_xor_f(bv, 32);
        const int oi = shfl_xor_i(bi, 32);
        if (better(ov, oi, bv, bi)) {
          bv = ov;
          bi = oi;
        }
        if (better(bv, bi, bestv[nb], besti[nb])) {
          bestv[nb] = bv;
          besti[nb] = bi;
        }
        if (logits) {
          const int n = 32 * nb + c;
          if (n < N)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              const int r = v0 + 8 * (j / 4) + 4 * u + (j % 4);
              if (r < V) logits[(size_t)n * V + r] = acc[nb][j];
            }
        }
      }
    }
  }
  if (u == 0)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) red[wave][32 * nb + c] = Cand{bestv[nb], besti[nb]};
  __syncthreads();
  for (int n = threadIdx.x; n < N; n += 256) {
    Cand b = red[0][n];
    for (int w2 = 1; w2 < 4; ++w2)
      if (better(red[w2][n].v, red[w2][n].i, b.v, b.i)) b = red[w2][n];
    partial[(size_t)blockIdx.x * N + n] = b;
  }
}

// Packed weight layout: for tile t (128 rows) and chunk kc (64 columns), the
// 16 KiB block at ((t * chunks + kc) * 128 + r) * 64 elements holds row
// t*128 + r; its physical 16-byte piece p holds columns
// kc*64 + 8*(p ^ (r/2)%8) .. +8, the swizzle the kernel's LDS reads expect.
// Rows >= V are zero.
__global__ __launch_bounds__(256) void lmhead_pack_kernel(const uint16_t* __restrict__ W, int V, int H,
                                                          uint16_t* __restrict__ out, long long pieces) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= pieces) return;
  const int chunks = H / 64;
  const int p = (int)(i % 8);
  const int r = (int)((i / 8) % kLmRows);
  const long long tk = i / (8 * kLmRows);  // t * chunks + kc
  const int kc = (int)(tk % chunks);
  const long long t = tk / chunks;
  const long long row = t * kLmRows + r;
  u32x4 v = {0, 0, 0, 0};
  if (row < V) v = ld16(W + row * H + kc * 64 + ((p ^ piece_swz(r)) * 8));
  st16(out + i * 8, v);
}

// float32 path: one thread per vocabulary row, one block column per node.
__global__ __launch_bounds__(256) void lmhead_f32_kernel(const float* __restrict__ X, const float* __restrict__ Wt,
                                                         int N, int H, int V, Cand* __restrict__ partial,
                                                         float* __restrict__ logits) {
  __shared__ Cand red[256];
  const int n = blockIdx.y;
  const int r = blockIdx.x * 256 + threadIdx.x;
  float acc = -INFINITY;
  if (r < V) {
    const f32x4* w4 = reinterpret_cast<const f32x4*>(Wt + (size_t)r * H);
    const f32x4* x4 = reinterpret_cast<const f32x4*>(X + (size_t)n * H);
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < H / 4; ++k) s += w4[k] * x4[k];
    acc = (s[0] + s[1]) + (s[2] + s[3]);
    if (logits) logits[(size_t)n * V + r] = acc;
  }
  red[threadIdx.x] = Cand{acc, r < V ? r : 0x7FFFFFFF};
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      const Cand o = red[threadIdx.x + off];
      if (better(o.v, o.i, red[threadIdx.x].v, red[threadIdx.x].i)) red[threadIdx.x] = o;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[(size_t)blockIdx.x * N + n] = red[0];
}

// One block per node: best of the per-block winners.
__global__ __launch_bounds__(256) void lmhead_finalize_kernel(const Cand* __restrict__ partial, int blocks, int N,
                                                              int32_t* __restrict__ ids, float* __restrict__ maxv) {
  __shared__ Cand red[256];
  const int n = blockIdx.x;
  Cand b{-INFINITY, 0x7FFFFFFF};
  for (int i = threadIdx.x; i < blocks; i += 256) {
    const Cand o = partial[(size_t)i * N + n];
    if (better(o.v, o.i, b.v, b.i)) b = o;
  }
  red[threadIdx.x] = b;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      const Cand o = red[threadIdx.x + off];
      if (better(o.v, o.i, red[threadIdx.x].v, red[threadIdx.x].i)) red[threadIdx.x] = o;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    ids[n] = red[0].i;
    maxv[n] = red[0].v;
  }
}

struct LmPlan {
  int nb, blocks;
  size_t ws_bytes;
};

LmPlan lm_plan(int N, int H, int V, ooo_dtype dt) {
  LmPlan p{};
  if (dt == OOO_BF16) {
    p.nb = N <= 32 ? 1 : N <= 64 ? 2 : N <= 128 ? 4 : 8;
    const int tiles = (V + kLmRows - 1) / kLmRows;
    p.blocks = tiles < device_cus() ? tiles : device_cus();  // persistent grid: one block per CU
  } else {
    p.blocks = (V + 255) / 256;
  }
  p.ws_bytes = (size_t)p.blocks * N * sizeof(Cand);
  return p;
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" size_t ooo_lmhead_workspace(int32_t n_nodes, int32_t hidden_dim, int32_t vocab, ooo_dtype dt) {
  if (n_nodes < 1 || hidden_dim < 1 || vocab < 1) return 0;
  return lm_plan(n_nodes, hidden_dim, vocab, dt).ws_bytes;
}

extern "C" size_t ooo_lmhead_packed_bytes(int32_t vocab, int32_t hidden_dim, ooo_dtype dt) {
  if (vocab < 1 || hidden_dim < 1 || hidden_dim % 64 || dt != OOO_BF16) return 0;
  const size_t tiles = (vocab + kLmRows - 1) / kLmRows;
  return tiles * kLmRows * (size_t)hidden_dim * 2;
}

extern "C" int ooo_lmhead_pack(const void* weight, int32_t vocab, int32_t hidden_dim, ooo_dtype dt, void* packed,
                               size_t packed_bytes, void* stream) {
  OOO_REQUIRE(weight && packed, OOO_ERR_INVALID, "ooo_lmhead_pack: null pointer");
  OOO_REQUIRE(vocab >= 1 && hidden_dim >= 1, OOO_ERR_INVALID, "ooo_lmhead_pack: sizes must be positive");
  OOO_REQUIRE(dt == OOO_BF16, OOO_ERR_UNSUPPORTED, "ooo_lmhead_pack: only OOO_BF16 weights are packed");
  OOO_REQUIRE(hidden_dim % 64 == 0, OOO_ERR_UNSUPPORTED, "ooo_lmhead_pack: hidden_dim %% 64 != 0");
  const size_t need = ooo_lmhead_packed_bytes(vocab, hidden_dim, dt);
  OOO_REQUIRE(packed_bytes >= need, OOO_ERR_CAPACITY, "ooo_lmhead_pack: %zu bytes needed (got %zu)", need,
              packed_bytes);
  const long long pieces = (long long)(need / 16);
  lmhead_pack_kernel<<<(unsigned)((pieces + 255) / 256), 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      (const uint16_t*)weight, vocab, hidden_dim, (uint16_t*)packed, pieces);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_lmhead_pack: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_lmhead_argmax(const void* hidden, const void* weight, int32_t n_nodes, int32_t hidden_dim,
                                 int32_t vocab, ooo_dtype dt, int32_t weight_layout, int32_t* argmax_ids,
                                 float* max_logit, float* logits, void* workspace, size_t ws_bytes, void* stream) {
  OOO_REQUIRE(hidden && weight && argmax_ids && max_logit, OOO_ERR_INVALID, "ooo_lmhead_argmax: null pointer");
  OOO_REQUIRE(n_nodes >= 1 && hidden_dim >= 1 && vocab >= 1, OOO_ERR_INVALID,
              "ooo_lmhead_argmax: sizes must be positive (n_nodes=%d hidden_dim=%d vocab=%d)", n_nodes,
              hidden_dim, vocab);
  OOO_REQUIRE(dt == OOO_F32 || dt == OOO_BF16, OOO_ERR_INVALID, "ooo_lmhead_argmax: unknown dtype %d", (int)dt);
  OOO_REQUIRE(weight_layout == OOO_W_ROWS || weight_layout == OOO_W_PACKED, OOO_ERR_INVALID,
              "ooo_lmhead_argmax: unknown weight layout %d", weight_layout);
  if (dt == OOO_BF16) {
    OOO_REQUIRE(hidden_dim % 64 == 0, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: bf16 needs hidden_dim %% 64 == 0");
    OOO_REQUIRE(n_nodes <= 256, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: bf16 supports up to 256 nodes");
  } else {
    OOO_REQUIRE(hidden_dim % 4 == 0, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: f32 needs hidden_dim %% 4 == 0");
    OOO_REQUIRE(n_nodes <= 65535, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: too many nodes");
    OOO_REQUIRE(weight_layout == OOO_W_ROWS, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: f32 weights are row-major only");
  }
  const LmPlan p = lm_plan(n_nodes, hidden_dim, vocab, dt);
  OOO_REQUIRE(workspace && ws_bytes >= p.ws_bytes, OOO_ERR_CAPACITY,
              "ooo_lmhead_argmax: workspace of %zu bytes needed (got %zu)", p.ws_bytes, ws_bytes);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  Cand* part = reinterpret_cast<Cand*>(workspace);
  if (dt == OOO_BF16) {
    const uint16_t* X = (const uint16_t*)hidden;
    const uint16_t* W = (const uint16_t*)weight;
    const bool pk = weight_layout == OOO_W_PACKED;
#define OOO_LM_LAUNCH(NBV)                                                                                   \
  do {                                                                                                      \
    if (pk)                                                                                                 \
      lmhead_bf16_kernel<NBV, true><<<p.blocks, kStreamThreads, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits); \
    else                                                                                                    \
      lmhead_bf16_kernel<NBV, false><<<p.blocks, kStreamThreads, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits); \
  } while (0)
    if (p.nb == 1) OOO_LM_LAUNCH(1);
    else if (p.nb == 2) OOO_LM_LAUNCH(2);
    else if (p.nb == 4) OOO_LM_LAUNCH(4);
    else OOO_LM_LAUNCH(8);
#undef OOO_LM_LAUNCH
  } else {
    lmhead_f32_kernel<<<dim3(p.blocks, n_nodes), 256, 0, st>>>((const float*)hidden, (const float*)weight, n_nodes,
                                                              hidden_dim, vocab, part, logits);
  }
  lmhead_finalize_kernel<<<n_nodes, 256, 0, st>>>(part, p.blocks, n_nodes, argmax_ids, max_logit);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_lmhead_argmax: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
