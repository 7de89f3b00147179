// LM head and greedy token of every trie node (Eq. 1: the next committed
// token is the target's most likely one; ties go to the lowest index).
//
// bf16 path: the product is W[V][H] x X[N][H]^T, a skinny GEMM that streams
// W from HBM once.  Each wave owns 32*RA vocabulary rows and all nodes in
// 32*NB columns, accumulating logits^T tiles on the matrix cores:
//  * A operand = W rows, B operand = X rows, both read straight from global
//    memory into registers (X is small and stays in L1/L2).
//  * The contraction index is permuted inside each 64-element chunk so a
//    lane reads 64 contiguous bytes of its row per chunk: MFMA k-step s,
//    lane half u, element e covers k = 32u + 8s + e.  The sum over k does
//    not depend on the order, and A and B use the same permutation.
//  * Chunks are double-buffered in registers so the next chunk's loads are
//    in flight while the current one is multiplied.
//  * Each lane ends with 16*RA logits of one node; the per-node argmax is
//    reduced in registers, across the two lane halves, across the block's
//    waves in LDS, and across blocks by a small finalize kernel reading the
//    per-block winners (deterministic: value, then lowest index).
#include <math.h>

#include "device_common.h"
#include "ooo_internal.h"

namespace ooo {
namespace {

struct Cand {
  float v;
  int i;
};

template <int RA, int NB>
__global__ __launch_bounds__(256) void lmhead_bf16_kernel(const uint16_t* __restrict__ X,
                                                          const uint16_t* __restrict__ Wt, int N, int H,
                                                          int V, Cand* __restrict__ partial,
                                                          float* __restrict__ logits) {
  constexpr int ROWS = 4 * 32 * RA;  // rows per block
  __shared__ Cand red[4][32 * NB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 31, u = lane >> 5;
  const int v0 = blockIdx.x * ROWS + wave * 32 * RA;

  const uint16_t* wp[RA];
  const uint16_t* xp[NB];
#pragma unroll
  for (int ra = 0; ra < RA; ++ra) {
    int r = v0 + 32 * ra + c;
    r = r < V ? r : V - 1;
    wp[ra] = Wt + (size_t)r * H + 32 * u;
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    int n = 32 * nb + c;
    n = n < N ? n : N - 1;
    xp[nb] = X + (size_t)n * H + 32 * u;
  }

  f32x16 acc[RA][NB];
#pragma unroll
  for (int ra = 0; ra < RA; ++ra)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[ra][nb] = f32x16{};

  u32x4 wa[RA][4], xa[NB][4], wb[RA][4], xb[NB][4];
  auto load = [&](u32x4 (&w)[RA][4], u32x4 (&x)[NB][4], int k0) {
#pragma unroll
    for (int ra = 0; ra < RA; ++ra)
#pragma unroll
      for (int s = 0; s < 4; ++s) w[ra][s] = ld16(wp[ra] + k0 + 8 * s);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int s = 0; s < 4; ++s) x[nb][s] = ld16(xp[nb] + k0 + 8 * s);
  };
  auto mma = [&](u32x4 (&w)[RA][4], u32x4 (&x)[NB][4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int ra = 0; ra < RA; ++ra)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[ra][nb] = mfma32(as_bf16x8(w[ra][s]), as_bf16x8(x[nb][s]), acc[ra][nb]);
  };

  const int chunks = H / 64;
  load(wa, xa, 0);
  int kc = 0;
  for (; kc + 2 <= chunks; kc += 2) {
    load(wb, xb, (kc + 1) * 64);
    mma(wa, xa);
    if (kc + 2 < chunks) load(wa, xa, (kc + 2) * 64);
    mma(wb, xb);
  }
  if (kc < chunks) mma(wa, xa);

  // acc[ra][nb][j]: vocabulary row v0 + 32ra + 8(j/4) + 4u + j%4, node 32nb + c
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int ra = 0; ra < RA; ++ra)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int r = v0 + 32 * ra + 8 * (j / 4) + 4 * u + (j % 4);
        const float val = acc[ra][nb][j];
        if (r < V && val > bv) {
          bv = val;
          bi = r;
        }
      }
    const float ov = shfl_xor_f(bv, 32);
    const int oi = shfl_xor_i(bi, 32);
    if (better(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
    if (u == 0) red[wave][32 * nb + c] = Cand{bv, bi};
  }
  if (logits) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int n = 32 * nb + c;
      if (n < N)
#pragma unroll
        for (int ra = 0; ra < RA; ++ra)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int r = v0 + 32 * ra + 8 * (j / 4) + 4 * u + (j % 4);
            if (r < V) logits[(size_t)n * V + r] = acc[ra][nb][j];
          }
    }
  }
  __syncthreads();
  for (int n = threadIdx.x; n < N && n < 32 * NB; n += blockDim.x) {
    Cand b = red[0][n];
    for (int w = 1; w < 4; ++w)
      if (better(red[w][n].v, red[w][n].i, b.v, b.i)) b = red[w][n];
    partial[(size_t)blockIdx.x * N + n] = b;
  }
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
  int ra, nb, rows, blocks;
  size_t ws_bytes;
};

LmPlan lm_plan(int N, int H, int V, ooo_dtype dt) {
  LmPlan p{};
  if (dt == OOO_BF16) {
    if (N <= 32) {
      p.ra = 4;
      p.nb = 1;
    } else if (N <= 64) {
      p.ra = 2;
      p.nb = 2;
    } else if (N <= 128) {
      p.ra = 2;
      p.nb = 4;
    } else {
      p.ra = 1;
      p.nb = 8;
    }
    p.rows = 128 * p.ra;
  } else {
    p.rows = 256;
  }
  p.blocks = (V + p.rows - 1) / p.rows;
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

extern "C" int ooo_lmhead_argmax(const void* hidden, const void* weight, int32_t n_nodes, int32_t hidden_dim,
                                 int32_t vocab, ooo_dtype dt, int32_t* argmax_ids, float* max_logit,
                                 float* logits, void* workspace, size_t ws_bytes, void* stream) {
  OOO_REQUIRE(hidden && weight && argmax_ids && max_logit, OOO_ERR_INVALID, "ooo_lmhead_argmax: null pointer");
  OOO_REQUIRE(n_nodes >= 1 && hidden_dim >= 1 && vocab >= 1, OOO_ERR_INVALID,
              "ooo_lmhead_argmax: sizes must be positive (n_nodes=%d hidden_dim=%d vocab=%d)", n_nodes,
              hidden_dim, vocab);
  OOO_REQUIRE(dt == OOO_F32 || dt == OOO_BF16, OOO_ERR_INVALID, "ooo_lmhead_argmax: unknown dtype %d", (int)dt);
  if (dt == OOO_BF16) {
    OOO_REQUIRE(hidden_dim % 64 == 0, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: bf16 needs hidden_dim %% 64 == 0");
    OOO_REQUIRE(n_nodes <= 256, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: bf16 supports up to 256 nodes");
  } else {
    OOO_REQUIRE(hidden_dim % 4 == 0, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: f32 needs hidden_dim %% 4 == 0");
    OOO_REQUIRE(n_nodes <= 65535, OOO_ERR_UNSUPPORTED, "ooo_lmhead_argmax: too many nodes");
  }
  const LmPlan p = lm_plan(n_nodes, hidden_dim, vocab, dt);
  OOO_REQUIRE(workspace && ws_bytes >= p.ws_bytes, OOO_ERR_CAPACITY,
              "ooo_lmhead_argmax: workspace of %zu bytes needed (got %zu)", p.ws_bytes, ws_bytes);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  Cand* part = reinterpret_cast<Cand*>(workspace);
  if (dt == OOO_BF16) {
    const uint16_t* X = (const uint16_t*)hidden;
    const uint16_t* W = (const uint16_t*)weight;
    if (p.nb == 1)
      lmhead_bf16_kernel<4, 1><<<p.blocks, 256, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits);
    else if (p.nb == 2)
      lmhead_bf16_kernel<2, 2><<<p.blocks, 256, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits);
    else if (p.nb == 4)
      lmhead_bf16_kernel<2, 4><<<p.blocks, 256, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits);
    else
      lmhead_bf16_kernel<1, 8><<<p.blocks, 256, 0, st>>>(X, W, n_nodes, hidden_dim, vocab, part, logits);
  } else {
    lmhead_f32_kernel<<<dim3(p.blocks, n_nodes), 256, 0, st>>>((const float*)hidden, (const float*)weight, n_nodes,
                                                              hidden_dim, vocab, part, logits);
  }
  lmhead_finalize_kernel<<<n_nodes, 256, 0, st>>>(part, p.blocks, n_nodes, argmax_ids, max_logit);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_lmhead_argmax: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
