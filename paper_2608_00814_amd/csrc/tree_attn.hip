// Tree-masked attention for one layer (Section 4.4: the target scores the
// whole candidate tree in one forward pass; node i sees the committed prefix
// and its own ancestors, exactly what sequential decoding of its path sees).
//
// bf16 path: split-KV flash-style kernel on gfx950 matrix cores.
//  * The G query heads that share a KV head are stacked with the nodes into
//    M = N*G query rows per KV head (row r = node r/G, head g*G + r%G), so
//    each K/V tile staged in LDS serves all of them.
//  * Work item = (KV head g, block of 32*WAVES rows, split s of the key
//    tiles).  Key tiles are 64 rows: the prefix tiles first, then the tree
//    tiles [P, P+N) where the ancestor bitmask is tested in registers.
//  * Scores are computed transposed, S^T = K Q^T, and the output as
//    O^T = V^T P^T.  With the A-operand rows of K permuted (bits 2 and 3 of
//    the row index swapped) every lane ends up holding one query row: its
//    softmax state, its probabilities (already in B-operand order for the
//    second product) and 16 of its output columns, so the online softmax
//    needs one cross-lane exchange per tile and no LDS round trip.
//  * V is transposed while it is staged (global -> registers -> LDS).
//  * Splits write float32 partials (unnormalised O, running max, sum) that
//    a second kernel combines; with one split the kernel writes O directly.
//  * Launch order is XCD-aware: consecutive work items (same KV head and
//    row block, neighbouring splits) go to blocks that share blockIdx % 8,
//    so one head's K/V stream stays in one XCD's L2.
#include <math.h>
#include <stdlib.h>

#include "device_common.h"
#include "ooo_internal.h"

namespace ooo {
namespace {

constexpr int kTile = 64;  // keys per tile

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  long long cap;
  int P, N;
  const uint64_t* mask;
  int W;
  int Hq, Hkv, G, M;
  float scale_log2e;
  uint16_t* out;
  float* part_o;
  float* part_ml;
  int splits, row_blocks, Mpad, tiles_prefix, tiles_total;
};

// swap bits 2 and 3: the K row a lane loads so that S^T lands with eight
// consecutive keys per lane and k-step
__device__ __forceinline__ int sigma(int c) { return (c & ~0xC) | ((c & 4) << 1) | ((c & 8) >> 1); }

template <int D, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void tree_attn_bf16_kernel(AttnArgs a) {
  constexpr int NT = 64 * WAVES;
  constexpr int BM = 32 * WAVES;
  constexpr int KLD = D + 8;       // K tile row stride (elements)
  constexpr int VLD = kTile + 8;   // V^T tile row stride (elements)
  constexpr int K_ELEMS = kTile * KLD;
  constexpr int V_ELEMS = D * VLD;
  constexpr int STAGE = K_ELEMS + V_ELEMS;
  constexpr int KCH = D / 8;                 // 16-byte chunks per row
  constexpr int K_ITEMS = kTile * KCH;
  constexpr int KI = K_ITEMS / NT;
  constexpr int V_ITEMS = (kTile / 4) * KCH; // (4-key group, chunk)
  constexpr int VI = (V_ITEMS + NT - 1) / NT;
  static_assert(K_ITEMS % NT == 0, "K staging must divide evenly");
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

  const int total = a.Hkv * a.row_blocks * a.splits;
  int w = blockIdx.x;
  if (total % 8 == 0) w = (w % 8) * (total / 8) + w / 8;
  const int s = w % a.splits;
  w /= a.splits;
  const int rb = w % a.row_blocks;
  const int g = w / a.row_blocks;
  const int t_begin = (int)((long long)s * a.tiles_total / a.splits);
  const int t_end = (int)((long long)(s + 1) * a.tiles_total / a.splits);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c = lane & 31, u = lane >> 5;
  const int row = rb * BM + wave * 32 + c;
  const bool row_ok = row < a.M;
  const int rr = row_ok ? row : a.M - 1;
  const int node = rr / a.G;
  const int head = g * a.G + (rr - node * a.G);

  bf16x8 qf[D / 16];
  {
    const uint16_t* qrow = a.q + ((size_t)node * a.Hq + head) * D;
#pragma unroll
    for (int dk = 0; dk < D / 16; ++dk) qf[dk] = as_bf16x8(ld16(qrow + 16 * dk + 8 * u));
  }
  const uint16_t* kbase = a.k + (size_t)g * a.cap * D;
  const uint16_t* vbase = a.v + (size_t)g * a.cap * D;

  u32x4 kreg[KI];
  u32x4 vreg[VI][4];

  auto tile_rows = [&](int t, int& row0, int& limit) {
    if (t < a.tiles_prefix) {
      row0 = t * kTile;
      limit = a.P;
    } else {
      row0 = a.P + (t - a.tiles_prefix) * kTile;
      limit = a.P + a.N;
    }
  };

  auto load_tile = [&](int t) {
    int row0, limit;
    tile_rows(t, row0, limit);
#pragma unroll
    for (int i = 0; i < KI; ++i) {
      const int item = tid + i * NT;
      const int r = item / KCH, ch = item % KCH;
      const int grow = row0 + r;
      kreg[i] = grow < limit ? ld16(kbase + (size_t)grow * D + ch * 8) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < VI; ++i) {
      const int item = tid + i * NT;
      const int kg = item % 16, dch = item / 16;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int grow = row0 + 4 * kg + r;
        vreg[i][r] = (item < V_ITEMS && grow < limit) ? ld16(vbase + (size_t)grow * D + dch * 8)
                                                       : u32x4{0, 0, 0, 0};
      }
    }
  };

  auto store_tile = [&](int stage) {
    uint16_t* Kl = lds + stage * STAGE;
    uint16_t* Vl = Kl + K_ELEMS;
#pragma unroll
    for (int i = 0; i < KI; ++i) {
      const int item = tid + i * NT;
      const int r = item / KCH, ch = item % KCH;
      st16(Kl + r * KLD + ch * 8, kreg[i]);
    }
#pragma unroll
    for (int i = 0; i < VI; ++i) {
      const int item = tid + i * NT;
      if (item < V_ITEMS) {
        const int kg = item % 16, dch = item / 16;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const uint32_t x0 = vreg[i][0][p], x1 = vreg[i][1][p], x2 = vreg[i][2][p], x3 = vreg[i][3][p];
          u32x2 even, odd;  // d = 8*dch + 2p (low halves) and + 1 (high halves)
          even[0] = (x0 & 0xFFFFu) | (x1 << 16);
          even[1] = (x2 & 0xFFFFu) | (x3 << 16);
          odd[0] = (x0 >> 16) | (x1 & 0xFFFF0000u);
          odd[1] = (x2 >> 16) | (x3 & 0xFFFF0000u);
          *reinterpret_cast<u32x2*>(Vl + (8 * dch + 2 * p) * VLD + 4 * kg) = even;
          *reinterpret_cast<u32x2*>(Vl + (8 * dch + 2 * p + 1) * VLD + 4 * kg) = odd;
        }
      }
    }
  };

  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  const int krow = sigma(c);

  if (t_begin < t_end) {
    load_tile(t_begin);
    store_tile(0);
  }
  __syncthreads();

  for (int t = t_begin; t < t_end; ++t) {
    const int stage = (t - t_begin) & 1;
    if (t + 1 < t_end) load_tile(t + 1);
    const uint16_t* Kl = lds + stage * STAGE;
    const uint16_t* Vl = Kl + K_ELEMS;

    // S^T = K Q^T for 64 keys x 32 rows (two 32-key halves)
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int dk = 0; dk < D / 16; ++dk) {
      const bf16x8 k0 = as_bf16x8(ld16(Kl + krow * KLD + 16 * dk + 8 * u));
      const bf16x8 k1 = as_bf16x8(ld16(Kl + (32 + krow) * KLD + 16 * dk + 8 * u));
      s0 = mfma32(k0, qf[dk], s0);
      s1 = mfma32(k1, qf[dk], s1);
    }
    // lane's value j of half h is key 32h + 16*(j/8) + 8u + j%8 of the tile
    float sv[32];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      sv[j] = s0[j] * a.scale_log2e;
      sv[16 + j] = s1[j] * a.scale_log2e;
    }
    int row0, limit;
    tile_rows(t, row0, limit);
    const bool tree = t >= a.tiles_prefix;
    if (tree || row0 + kTile > limit) {
      uint64_t mw = ~0ull;
      if (tree) {
        const int word = (row0 - a.P) / 64;
        mw = a.mask[(size_t)node * a.W + word];
      }
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const int off = 16 * (j / 8) + 8 * u + (j % 8);
        const bool ok = (row0 + off < limit) && ((mw >> off) & 1ull);
        if (!ok) sv[j] = -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 32; ++j) mx = fmaxf(mx, sv[j]);
    mx = fmaxf(mx, shfl_xor_f(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      sv[j] = exp2f(sv[j] - m_use);
      psum += sv[j];
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;

    bf16x8 pf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk[e] = pack_bf16x2(sv[8 * ks + 2 * e], sv[8 * ks + 2 * e + 1]);
      pf[ks] = as_bf16x8(pk);
    }
    // O^T += V^T P^T
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 vv = as_bf16x8(ld16(Vl + (32 * dt + c) * VLD + 16 * ks + 8 * u));
        oacc[dt] = mfma32(vv, pf[ks], oacc[dt]);
      }
    }
    if (t + 1 < t_end) store_tile(stage ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + shfl_xor_f(l_run, 32);
  if (!row_ok) return;
  // lane holds output columns d = 32*dt + 8*(j/4) + 4u + j%4 of its row
  if (a.splits == 1) {
    const float inv = 1.f / l_tot;
    uint16_t* orow = a.out + ((size_t)node * a.Hq + head) * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        u32x2 pk;
        pk[0] = pack_bf16x2(oacc[dt][4 * q4] * inv, oacc[dt][4 * q4 + 1] * inv);
        pk[1] = pack_bf16x2(oacc[dt][4 * q4 + 2] * inv, oacc[dt][4 * q4 + 3] * inv);
        *reinterpret_cast<u32x2*>(orow + 32 * dt + 8 * q4 + 4 * u) = pk;
      }
    }
  } else {
    const size_t prow = ((size_t)s * a.Hkv + g) * a.Mpad + row;
    float* po = a.part_o + prow * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 v4 = {oacc[dt][4 * q4], oacc[dt][4 * q4 + 1], oacc[dt][4 * q4 + 2], oacc[dt][4 * q4 + 3]};
        *reinterpret_cast<f32x4*>(po + 32 * dt + 8 * q4 + 4 * u) = v4;
      }
    }
    if (u == 0) {
      a.part_ml[prow * 2] = m_run;
      a.part_ml[prow * 2 + 1] = l_tot;
    }
  }
}

// Merge the splits of each query row: O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s.
template <int D>
__global__ __launch_bounds__(256) void tree_attn_combine_kernel(AttnArgs a) {
  constexpr int TPR = D / 4;  // threads per row, 4 columns each
  const int gr = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  if (gr >= a.Hkv * a.M) return;
  const int g = gr / a.M, r = gr % a.M;
  const int d0 = (threadIdx.x % TPR) * 4;
  float mmax = -INFINITY;
  for (int s = 0; s < a.splits; ++s) mmax = fmaxf(mmax, a.part_ml[(((size_t)s * a.Hkv + g) * a.Mpad + r) * 2]);
  float den = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < a.splits; ++s) {
    const size_t prow = ((size_t)s * a.Hkv + g) * a.Mpad + r;
    const float m = a.part_ml[prow * 2];
    if (m == -INFINITY) continue;
    const float wgt = exp2f(m - mmax);
    den += wgt * a.part_ml[prow * 2 + 1];
    acc += wgt * *reinterpret_cast<const f32x4*>(a.part_o + prow * D + d0);
  }
  const float inv = 1.f / den;
  const int node = r / a.G, head = g * a.G + r % a.G;
  u32x2 pk;
  pk[0] = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  pk[1] = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<u32x2*>(a.out + ((size_t)node * a.Hq + head) * D + d0) = pk;
}

// float32 path: one wave per (node, query head), keys walked in order with
// an online softmax; each lane owns head_dim/64 columns.
template <int D>
__global__ __launch_bounds__(64) void tree_attn_f32_kernel(const float* q, const float* k, const float* v,
                                                           long long cap, int P, int N, const uint64_t* mask,
                                                           int W, int Hq, int Hkv, float scale, float* out) {
  constexpr int C = D / 64;
  const int node = blockIdx.x / Hq, head = blockIdx.x % Hq;
  const int g = head / (Hq / Hkv);
  const int lane = threadIdx.x;
  float qv[C], o[C];
  for (int i = 0; i < C; ++i) {
    qv[i] = q[((size_t)node * Hq + head) * D + lane + 64 * i];
    o[i] = 0.f;
  }
  const float* kb = k + (size_t)g * cap * D;
  const float* vb = v + (size_t)g * cap * D;
  float m = -INFINITY, l = 0.f;
  auto visit = [&](int rowi) {
    float part = 0.f;
    for (int i = 0; i < C; ++i) part += qv[i] * kb[(size_t)rowi * D + lane + 64 * i];
    for (int off = 32; off > 0; off >>= 1) part += shfl_xor_f(part, off);
    const float sc = part * scale;
    const float m_new = fmaxf(m, sc);
    const float alpha = expf(m - m_new);
    const float p = expf(sc - m_new);
    l = l * alpha + p;
    for (int i = 0; i < C; ++i) o[i] = o[i] * alpha + p * vb[(size_t)rowi * D + lane + 64 * i];
    m = m_new;
  };
  for (int j = 0; j < P; ++j) visit(j);
  for (int j = 0; j < N; ++j)
    if ((mask[(size_t)node * W + j / 64] >> (j % 64)) & 1ull) visit(P + j);
  for (int i = 0; i < C; ++i) out[((size_t)node * Hq + head) * D + lane + 64 * i] = o[i] / l;
}

struct Plan {
  int waves, row_blocks, Mpad, tiles_prefix, tiles_total, splits;
  size_t ws_bytes;
};

Plan make_plan(int N, int Hq, int Hkv, int D, int P, ooo_dtype dt) {
  Plan p{};
  if (dt != OOO_BF16) return p;
  const int G = Hq / Hkv;
  const int M = N * G;
  p.waves = M <= 64 ? 2 : 4;
  const int BM = 32 * p.waves;
  p.row_blocks = (M + BM - 1) / BM;
  p.Mpad = p.row_blocks * BM;
  p.tiles_prefix = (P + kTile - 1) / kTile;
  p.tiles_total = p.tiles_prefix + (N + kTile - 1) / kTile;
  const int base = Hkv * p.row_blocks;
  int splits = (256 + base - 1) / base;
  if (const char* env = getenv("OOO_ATTN_SPLITS")) splits = atoi(env);
  if (splits > 32) splits = 32;
  if (splits > p.tiles_total) splits = p.tiles_total;
  if (splits < 1) splits = 1;
  p.splits = splits;
  if (splits > 1)
    p.ws_bytes = (size_t)splits * Hkv * p.Mpad * (size_t)D * sizeof(float) +
                 (size_t)splits * Hkv * p.Mpad * 2 * sizeof(float) + 256;
  return p;
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" size_t ooo_tree_attn_workspace(int32_t n_nodes, int32_t n_q_heads, int32_t n_kv_heads,
                                          int32_t head_dim, int32_t prefix_len, ooo_dtype dt) {
  if (n_nodes < 1 || n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads || prefix_len < 0) return 0;
  return make_plan(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt).ws_bytes;
}

extern "C" int ooo_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                             int32_t prefix_len, int32_t n_nodes, const uint64_t* anc_mask,
                             int32_t mask_words, int32_t n_q_heads, int32_t n_kv_heads,
                             int32_t head_dim, float scale, ooo_dtype dt, void* out, void* workspace,
                             size_t ws_bytes, void* stream) {
  OOO_REQUIRE(q && k_cache && v_cache && anc_mask && out, OOO_ERR_INVALID, "ooo_tree_attn: null pointer");
  OOO_REQUIRE(n_nodes >= 1, OOO_ERR_INVALID, "ooo_tree_attn: n_nodes must be >= 1");
  OOO_REQUIRE(prefix_len >= 0, OOO_ERR_INVALID, "ooo_tree_attn: prefix_len must be >= 0");
  OOO_REQUIRE(n_q_heads >= 1 && n_kv_heads >= 1 && n_q_heads % n_kv_heads == 0, OOO_ERR_INVALID,
              "ooo_tree_attn: n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)", n_q_heads,
              n_kv_heads);
  OOO_REQUIRE((int64_t)prefix_len + n_nodes <= cap, OOO_ERR_INVALID,
              "ooo_tree_attn: prefix_len + n_nodes (%lld) exceeds cap (%lld)",
              (long long)prefix_len + n_nodes, (long long)cap);
  OOO_REQUIRE(mask_words >= 1 && (int64_t)mask_words * 64 >= n_nodes && mask_words <= 16, OOO_ERR_INVALID,
              "ooo_tree_attn: mask_words=%d cannot describe %d nodes (max 16 words)", mask_words, n_nodes);
  OOO_REQUIRE(dt == OOO_F32 || dt == OOO_BF16, OOO_ERR_INVALID, "ooo_tree_attn: unknown dtype %d", (int)dt);
  OOO_REQUIRE(head_dim == 64 || head_dim == 128, OOO_ERR_UNSUPPORTED,
              "ooo_tree_attn: head_dim %d not supported (64 or 128)", head_dim);
  OOO_REQUIRE((int64_t)n_nodes * n_q_heads <= (1 << 30), OOO_ERR_UNSUPPORTED, "ooo_tree_attn: too many rows");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int G = n_q_heads / n_kv_heads;

  if (dt == OOO_F32) {
    const dim3 grid(n_nodes * n_q_heads);
    if (head_dim == 64)
      tree_attn_f32_kernel<64><<<grid, 64, 0, st>>>((const float*)q, (const float*)k_cache, (const float*)v_cache,
                                                    cap, prefix_len, n_nodes, anc_mask, mask_words, n_q_heads,
                                                    n_kv_heads, scale, (float*)out);
    else
      tree_attn_f32_kernel<128><<<grid, 64, 0, st>>>((const float*)q, (const float*)k_cache, (const float*)v_cache,
                                                     cap, prefix_len, n_nodes, anc_mask, mask_words, n_q_heads,
                                                     n_kv_heads, scale, (float*)out);
  } else {
    const Plan p = make_plan(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt);
    OOO_REQUIRE(ws_bytes >= p.ws_bytes && (p.ws_bytes == 0 || workspace), OOO_ERR_CAPACITY,
                "ooo_tree_attn: workspace of %zu bytes needed (got %zu)", p.ws_bytes, ws_bytes);
    AttnArgs a{};
    a.q = (const uint16_t*)q;
    a.k = (const uint16_t*)k_cache;
    a.v = (const uint16_t*)v_cache;
    a.cap = cap;
    a.P = prefix_len;
    a.N = n_nodes;
    a.mask = anc_mask;
    a.W = mask_words;
    a.Hq = n_q_heads;
    a.Hkv = n_kv_heads;
    a.G = G;
    a.M = n_nodes * G;
    a.scale_log2e = scale * 1.4426950408889634f;
    a.out = (uint16_t*)out;
    a.splits = p.splits;
    a.row_blocks = p.row_blocks;
    a.Mpad = p.Mpad;
    a.tiles_prefix = p.tiles_prefix;
    a.tiles_total = p.tiles_total;
    if (p.splits > 1) {
      a.part_o = (float*)workspace;
      a.part_ml = a.part_o + (size_t)p.splits * n_kv_heads * p.Mpad * head_dim;
    }
    const dim3 grid(n_kv_heads * p.row_blocks * p.splits);
    if (head_dim == 128) {
      if (p.waves == 2) tree_attn_bf16_kernel<128, 2><<<grid, 128, 0, st>>>(a);
      else tree_attn_bf16_kernel<128, 4><<<grid, 256, 0, st>>>(a);
    } else {
      if (p.waves == 2) tree_attn_bf16_kernel<64, 2><<<grid, 128, 0, st>>>(a);
      else tree_attn_bf16_kernel<64, 4><<<grid, 256, 0, st>>>(a);
    }
    if (p.splits > 1) {
      const int rows = n_kv_heads * a.M;
      const int rows_per_block = 256 / (head_dim / 4);
      const dim3 cgrid((rows + rows_per_block - 1) / rows_per_block);
      if (head_dim == 128) tree_attn_combine_kernel<128><<<cgrid, 256, 0, st>>>(a);
      else tree_attn_combine_kernel<64><<<cgrid, 256, 0, st>>>(a);
    }
  }
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_tree_attn: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
