// Tree-masked attention for one layer (Section 4.5: the target scores the
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

#include <type_traits>

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

typedef short i16x4 __attribute__((ext_vector_type(4)));
#define OOO_LDS(p) ((__attribute__((address_space(3))) void*)(p))
#define OOO_GLB(p) ((const __attribute__((address_space(1))) void*)(p))

// Workgroup barrier without the memory-model fence __syncthreads() adds: the
// fence would make the loader wave wait for every in-flight LDS DMA.  The
// "memory" clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt vmcnt(n) (n <= 63), leaving the other counters alone.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x0F70);
}

// LDS ring geometry for one head_dim.  A tile is 64 rows of K and 64 rows of
// V, each row D bf16 values = D/8 16-byte chunks, stored row-major with
// chunk c of row r at position c ^ (r % (D/8)).  One 1 KiB DMA instruction
// copies whole contiguous rows (coalesced in global memory); the XOR
// swizzle makes reads of one chunk down many rows hit distinct banks.  K
// tiles of all stages come first, then the V tiles, then the block's
// queries (padded rows, written once), so every LDS read is a per-lane
// offset plus a compile-time immediate below 64 KiB.
template <int D>
struct Ring {
  static constexpr int CH = D / 8;           // chunks per row
  static constexpr int ROWB = 2 * D;         // bytes per row
  static constexpr int MAT = kTile * ROWB;   // bytes of one K or V tile
  static constexpr int NS = 3;               // stages
  static constexpr int VREG = NS * MAT;      // start of the V tiles
  static constexpr int QREG = 2 * NS * MAT;  // start of the queries
  static constexpr int QLD = ROWB + 16;      // padded query row
  static constexpr int DMA_MAT = MAT / 1024; // DMA instructions per matrix
  static constexpr int RPI = 1024 / ROWB;    // rows per DMA instruction
  static_assert(2 * DMA_MAT <= 63, "vmcnt range");
};

template <int D, int CW>
__global__ __launch_bounds__(64 * (CW + 2)) __attribute__((amdgpu_waves_per_eu(1, 2)))
void tree_attn_bf16_kernel(AttnArgs a) {
  using R = Ring<D>;
  constexpr int BM = 32 * CW;  // query rows per block
  __shared__ __attribute__((aligned(1024))) uint8_t lds[R::QREG + BM * R::QLD];

  const int total = a.Hkv * a.row_blocks * a.splits;
  int w = blockIdx.x;
  if (total % 8 == 0) w = (w % 8) * (total / 8) + w / 8;
  const int s = w % a.splits;
  w /= a.splits;
  const int rb = w % a.row_blocks;
  const int g = w / a.row_blocks;
  const int t_begin = (int)((long long)s * a.tiles_total / a.splits);
  const int t_end = (int)((long long)(s + 1) * a.tiles_total / a.splits);
  const int ntiles = t_end - t_begin;  // >= 1 because splits <= tiles

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  if (wave >= CW) {
    // ------------------------------------------------- loaders: K (CW), V (CW+1)
    const bool is_v = wave == CW + 1;
    const uint16_t* src = (is_v ? a.v : a.k) + (size_t)g * a.cap * D;
    uint8_t* dst0 = lds + (is_v ? R::VREG : 0);
    auto issue = [&](int t, int stage) {
      int row0, limit;
      if (t < a.tiles_prefix) {
        row0 = t * kTile;
        limit = a.P;
      } else {
        row0 = a.P + (t - a.tiles_prefix) * kTile;
        limit = a.P + a.N;
      }
      uint8_t* dst = dst0 + stage * R::MAT;
#pragma unroll
      for (int j = 0; j < R::DMA_MAT; ++j) {
        // lane = (row within the instruction, swizzled chunk); rows past the
        // limit re-read the last valid row (masked keys, zero probability)
        const int r = j * R::RPI + lane / R::CH;
        const int c = (lane % R::CH) ^ (r % R::CH);
        const size_t off = (size_t)min(row0 + r, limit - 1) * D + c * 8;
        __builtin_amdgcn_global_load_lds(OOO_GLB(src + off), OOO_LDS(dst + j * 1024), 16, 0, 0);
      }
    };
    issue(t_begin, 0);
    if (ntiles > 1) issue(t_begin + 1, 1);
    for (int i = 0; i < ntiles; ++i) {
      if (i + 1 < ntiles) wait_vmcnt<R::DMA_MAT>();  // tile i landed, i+1 may be in flight
      else wait_vmcnt<0>();
      wg_barrier();
      if (i + 2 < ntiles) issue(t_begin + i + 2, (i + 2) % R::NS);
    }
    return;
  }

  // ------------------------------------------------------------------ compute
  const int c = lane & 31, u = lane >> 5;
  const int row = rb * BM + wave * 32 + c;
  const bool row_ok = row < a.M;
  const int rr = row_ok ? row : a.M - 1;
  const int node = rr / a.G;
  const int head = g * a.G + (rr - node * a.G);

  // this wave's 32 query rows into its private LDS slice (padded rows)
  const uint32_t qb = R::QREG + (wave * 32 + c) * R::QLD + u * 16;  // + 32*dk
  {
    const uint16_t* qrow = a.q + ((size_t)node * a.Hq + head) * D;
#pragma unroll
    for (int dk = 0; dk < D / 16; ++dk)
      *reinterpret_cast<u32x4*>(lds + qb + 32 * dk) = ld16(qrow + 16 * dk + 8 * u);
  }
  // ancestor-mask word of the next tree tile this split will see
  int next_tt = t_begin > a.tiles_prefix ? t_begin - a.tiles_prefix : 0;
  uint64_t mnext = a.mask[(size_t)node * a.W + next_tt];

  // per-lane LDS byte offsets (loop invariant).  K fragment (half kt, k-step
  // dk): chunk 2dk+u of row sigma(c)+32kt.  V^T transpose-read source (for
  // column block dt, key step ks, half h): row 16ks+4h+8(g16/2)+li/4, columns
  // 32dt+16(g16%2)+4(li%4) .. +3.
  const int krow = sigma(c);
  uint32_t koff[D / 16];
#pragma unroll
  for (int dk = 0; dk < D / 16; ++dk) koff[dk] = krow * R::ROWB + (((2 * dk + u) ^ (krow % R::CH)) << 4);
  const int g16 = lane >> 4, li = lane & 15;
  uint32_t voff[D / 32][2];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int vr = 4 * h + 8 * (g16 >> 1) + (li >> 2);  // key row within a 16-row block
      const int col = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
      voff[dt][h] = R::VREG + vr * R::ROWB + (((col >> 3) ^ (vr % R::CH)) << 4) + (col & 7) * 2;
    }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  auto tile = [&](int i, auto stage_c) {
    constexpr int ST = decltype(stage_c)::value;
    const int t = t_begin + i;
    wg_barrier();  // tile t is in stage ST
    const uint8_t* Ks = lds + ST * R::MAT;

    // S^T = K Q^T for both 32-key halves first, so the softmax of half A
    // (VALU) can run while the matrix cores still work on half B.
    f32x16 sh[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int b4 = 0; b4 < D / 64; ++b4) {
      bf16x8 k0[4], k1[4], qq[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int dk = 4 * b4 + j;
        qq[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(lds + qb + 32 * dk));
        k0[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(Ks + koff[dk]));
        k1[j] = as_bf16x8(*reinterpret_cast<const u32x4*>(Ks + koff[dk] + 32 * R::ROWB));
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        sh[0] = mfma32(k0[j], qq[j], sh[0]);
        sh[1] = mfma32(k1[j], qq[j], sh[1]);
      }
    }
    const bool tree = t >= a.tiles_prefix;
    const int row0 = tree ? a.P + (t - a.tiles_prefix) * kTile : t * kTile;
    const int limit = tree ? a.P + a.N : a.P;
    const bool masked = tree || row0 + kTile > limit;
    uint64_t mw = ~0ull;
    if (tree) {
      mw = mnext;
      next_tt = min(next_tt + 1, a.W - 1);
      mnext = a.mask[(size_t)node * a.W + next_tt];
    }

#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      // lane's value j of this half is key 32hf + 16*(j/8) + 8u + j%8 of the tile
      float sv[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) sv[j] = sh[hf][j];
      if (masked) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int off = 32 * hf + 16 * (j / 8) + 8 * u + (j % 8);
          const bool ok = (row0 + off < limit) && ((mw >> off) & 1ull);
          if (!ok) sv[j] = -INFINITY;
        }
      }
      float mx = sv[0];
#pragma unroll
      for (int j = 1; j < 16; ++j) mx = __builtin_fmaxf(mx, sv[j]);
      {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = __builtin_fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * a.scale_log2e;  // log2 units
      }
      // Lazy rescaling: the reference max m_run moves only when some row of
      // the wave grows by more than 2^8, so probabilities stay <= 256 (fine
      // for fp32 sums and bf16 operands) and O, l are rescaled rarely.
      if (__any(mx > m_run + 8.f)) {
        const float m_new = __builtin_fmaxf(m_run, mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
        m_run = m_new;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      float psum = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        sv[j] = __builtin_amdgcn_exp2f(fmaf(sv[j], a.scale_log2e, -m_use));
        psum += sv[j];
      }
      l_run += psum;
      bf16x8 pf[2];
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        u32x4 pk;
#pragma unroll
        for (int e = 0; e < 4; ++e) pk[e] = pack_bf16x2(sv[8 * k2 + 2 * e], sv[8 * k2 + 2 * e + 1]);
        pf[k2] = as_bf16x8(pk);
      }
      // O^T += V^T P^T for this half (key steps ks = 2hf, 2hf+1).  V^T
      // fragments come from the row-major V tile through the LDS transpose
      // read: within each 16-lane group, source lane 4k+q points at key row
      // k, columns 4q..4q+3, and lane i receives column i of the four rows.
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        const int ks = 2 * hf + k2;
        bf16x8 vv[D / 32];
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          u32x2 lohi[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint8_t* p = lds + voff[dt][h] + ST * R::MAT + ks * 16 * R::ROWB;
            lohi[h] = __builtin_bit_cast(
                u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((i16x4 __attribute__((address_space(3)))*)OOO_LDS(p)));
          }
          vv[dt] = as_bf16x8(u32x4{lohi[0][0], lohi[0][1], lohi[1][0], lohi[1][1]});
        }
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = mfma32(vv[dt], pf[k2], oacc[dt]);
      }
    }
  };
  int i = 0;
  for (; i + R::NS <= ntiles; i += R::NS) {
    tile(i, std::integral_constant<int, 0>{});
    tile(i + 1, std::integral_constant<int, 1>{});
    tile(i + 2, std::integral_constant<int, 2>{});
  }
  if (i < ntiles) tile(i, std::integral_constant<int, 0>{});
  if (i + 1 < ntiles) tile(i + 1, std::integral_constant<int, 1>{});

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

// Merge the splits of each query row, online over the splits:
// O = sum_s 2^(m_s - m) O_s / sum_s 2^(m_s - m) l_s.  A split that saw no
// allowed key has m_s = -inf, l_s = 0 and O_s = 0 and gets weight zero.
// Every split's loads are independent of the running state, so the unrolled
// loop keeps many of them in flight.
template <int D>
__global__ __launch_bounds__(256) void tree_attn_combine_kernel(AttnArgs a) {
  constexpr int TPR = D / 4;  // threads per row, 4 columns each
  const int gr = blockIdx.x * (256 / TPR) + threadIdx.x / TPR;
  if (gr >= a.Hkv * a.M) return;
  const int g = gr / a.M, r = gr % a.M;
  const int d0 = (threadIdx.x % TPR) * 4;
  const size_t stride = (size_t)a.Hkv * a.Mpad;  // rows between consecutive splits
  const size_t row0 = (size_t)g * a.Mpad + r;
  float mrun = -INFINITY, den = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int s = 0; s < a.splits; ++s) {
    const size_t prow = row0 + s * stride;
    const float m = a.part_ml[prow * 2], l = a.part_ml[prow * 2 + 1];
    const f32x4 o = *reinterpret_cast<const f32x4*>(a.part_o + prow * D + d0);
    const float mn = __builtin_fmaxf(mrun, m);
    const float base = mn == -INFINITY ? 0.f : mn;
    const float c_old = __builtin_amdgcn_exp2f(mrun - base), c_new = __builtin_amdgcn_exp2f(m - base);
    den = den * c_old + l * c_new;
    acc = acc * c_old + o * c_new;
    mrun = mn;
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
      if (p.waves == 2) tree_attn_bf16_kernel<128, 2><<<grid, 256, 0, st>>>(a);
      else tree_attn_bf16_kernel<128, 4><<<grid, 384, 0, st>>>(a);
    } else {
      if (p.waves == 2) tree_attn_bf16_kernel<64, 2><<<grid, 256, 0, st>>>(a);
      else tree_attn_bf16_kernel<64, 4><<<grid, 384, 0, st>>>(a);
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
