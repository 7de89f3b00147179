// Projections of the target decoder around the verification path: the
// q/k/v, output and MLP projections of every layer (Section 4.5: the target
// scores the tree in one forward pass; Section 5: Qwen3 targets).  With the
// trie's N <= 256 rows these are skinny GEMMs, Y[N][O] = X[N][K] W[O][K]^T,
// bound by streaming W from HBM once.
//
// Design (the LM head's streaming scheme, made shape-independent):
//  * W is packed once into 16 KiB blocks of 128 rows x 64 columns (the LM
//    head's layout, ooo_linear_pack); the work is the sequence of (128-row
//    tile, 64-column chunk) blocks in tile-major order.
//  * Stream-K: a persistent grid (one block per CU) where block b takes the
//    contiguous run of chunks [C b / B, C (b + 1) / B).  Every block streams
//    the same number of bytes whatever O and K are; a run covers the end of
//    one tile and the start of the next.
//  * Inside a block, the LM head's streaming core (stream_core.h): two
//    loader waves DMA the W chunk (two 32-row slots each) and a third the X
//    chunk into an LDS ring; four compute waves run mfma_f32_32x32x16_bf16
//    (32 W rows x the nodes each).
//  * At the end of each tile segment a block stores its partial sums in the
//    workspace as fp16 ([node][128 rows]) times a power of two per compute
//    wave (its 32 rows), chosen so that the wave's largest magnitude lies
//    in [2^14, 2^15): half the bytes of fp32, with the range of fp32.  A
//    reduce kernel adds a tile's partials in float32 in block order
//    (deterministic, no atomics) and applies the epilogue: store fp32 or
//    bf16, add into an fp32 output (the residual rows), or silu(gate) * up
//    of a fused gate/up projection.
#include <math.h>

#include <vector>

#include "device_common.h"
#include "ooo_internal.h"
#include "rope.h"
#include "stream_core.h"

namespace ooo {
namespace {

constexpr int kRows = kStreamRows;  // W rows per tile (4 compute waves x 32)

// Stream-K partial sums in the workspace: slot k (block b, segment j: k =
// b * seg + j) holds v[k][node][128 rows] in fp16 and sc[k][4], the factor
// that turns the fp16 values of rows 32 w .. 32 w + 31 back into the sums.
struct Partials {
  uint16_t* v;
  float* sc;
};

// first chunk of block b's run
__host__ __device__ __forceinline__ long long run_lo(long long C, int b, int B) { return C * b / B; }

template <int NB, bool PACKED>
__global__ __launch_bounds__(kStreamThreads) void linear_bf16_kernel(const uint16_t* __restrict__ X,
                                                          const uint16_t* __restrict__ Wt, int N, int K, int O,
                                                          int seg_per_block, Partials part) {
  using R = StreamRing<NB>;
  constexpr int NPAD = 32 * NB;
  __shared__ __attribute__((aligned(1024))) uint8_t lds[R::BYTES];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int KC = K / 64;
  const int tiles = (O + kRows - 1) / kRows;
  const long long C = (long long)tiles * KC;
  const int b = (int)blockIdx.x, B = (int)gridDim.x;
  const long long lo = run_lo(C, b, B);
  const int total = (int)(run_lo(C, b + 1, B) - lo);  // chunks of this block (>= 1: B <= C)
  const int first_tile = (int)(lo / KC);

  if (wave >= 4) {
    // ------------------------------------------ loaders: W rows 0-63 (4), 64-127 (5), X (6)
    const bool is_x = wave == 6;
    const int half = wave - 4;
    // (tile, chunk) of the next chunk to issue; issues come in order
    int it = first_tile, ikc = (int)(lo - (long long)first_tile * KC);
    auto issue = [&](int q, int stage) {
      const int t = it, kc = ikc;
      if (++ikc == KC) {
        ikc = 0;
        ++it;
      }
      if (!is_x) {
        // this loader's slots 2 half, 2 half + 1: tile rows 64 half .. +63
        uint8_t* dst = lds + stage * R::WS + half * (R::WS / 2);
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
          const int s4 = 2 * half + sl;
          if (PACKED)
            dma_w_slot_packed(Wt + (((size_t)t * KC + kc) * kRows + 32 * s4) * 64 + lane * 8, 1, dst + sl * 4096);
          else
            dma_w_slot_rows(Wt, K, t * kRows + 32 * s4, O, kc, dst + sl * 4096, lane);
        }
      } else {
        dma_x_chunk<NB>(X, N, K, kc, lds + R::XREG + stage * R::XS, lane);
      }
    };
    if (is_x) loader_stream<R::NS, R::XDMA>(total, issue);
    else loader_stream<R::NS, R::WDMA>(total, issue);
    return;
  }

  // ------------------------------------------------------------------ compute
  const int c = lane & 31, u = lane >> 5;
  uint32_t off[4];
  frag_offsets(lane, off);
  const uint32_t wrow = wave * 32 * 128;
  f32x16 acc[NB];
  int t = first_tile, kc = (int)(lo - (long long)first_tile * KC) - 1;
  for (int q = 0; q < total; ++q) {
    if (++kc == KC) {
      kc = 0;
      ++t;
    }
    if (q == 0 || kc == 0) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x16{};
    }
    const int stage = q % R::NS;
    wg_barrier();
    chunk_mfma<NB>(lds + stage * R::WS + wrow, lds + R::XREG + stage * R::XS, off, acc);
    if (q == total - 1 || kc == KC - 1) {
      // segment done: acc[nb][j] = partial of tile row wave*32 + 8(j/4) + 4u + j%4, node 32nb + c.
      // Scale: the wave's largest finite magnitude a < 2^ex goes to
      // [2^14, 2^15) (fp16 holds up to 65504); exact powers of two both
      // ways.  Inf and NaN stay what they are and do not set the scale.
      float amax = 0.f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float m = __builtin_fabsf(acc[nb][j]);
          amax = __builtin_fmaxf(amax, m < INFINITY ? m : 0.f);
        }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) amax = __builtin_fmaxf(amax, shfl_xor_f(amax, o));
      const int ex = min(max(__builtin_amdgcn_frexp_expf(amax), -100), 100);
      const float mul = __builtin_amdgcn_ldexpf(1.f, 15 - ex);
      const size_t slot = (size_t)b * seg_per_block + (t - first_tile);
      uint16_t* dst = part.v + slot * NPAD * kRows;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq)
          *reinterpret_cast<u32x2*>(dst + (size_t)(32 * nb + c) * kRows + wave * 32 + 8 * jq + 4 * u) =
              u32x2{pack_f16x2(acc[nb][4 * jq] * mul, acc[nb][4 * jq + 1] * mul),
                    pack_f16x2(acc[nb][4 * jq + 2] * mul, acc[nb][4 * jq + 3] * mul)};
      if (lane == 0) part.sc[slot * 4 + wave] = __builtin_amdgcn_ldexpf(1.f, ex - 15);
    }
  }
}

enum Epi { kStoreF32 = 0, kStoreBF16 = 1, kAddF32 = 2, kSwiGLU = 3 };

// Workspace slots holding tile t's partials, in block order (the blocks
// whose runs intersect the tile's chunks [t KC, (t + 1) KC)); returns the
// count.  Called by one thread per reduce block.
__device__ int tile_slots(long long C, int B, int KC, int seg, int t, int* slots) {
  if (C * B < (1LL << 31)) {
    // Every product below fits in 32 bits (g0 <= C, b <= B), and 32-bit
    // divisions cost a small fraction of the emulated 64-bit ones: the same
    // slot list, computed several times faster.
    const unsigned c = (unsigned)C, bb = (unsigned)B;
    const auto lo = [&](int b) { return (int)(c * (unsigned)b / bb); };
    const int g0 = t * KC, g1 = g0 + KC;
    int b = (int)((unsigned)g0 * bb / c);
    while (b + 1 < B && lo(b + 1) <= g0) ++b;
    while (b > 0 && lo(b) > g0) --b;
    int n = 0;
    for (; b < B; ++b) {
      const int l = lo(b);
      if (l >= g1) break;
      slots[n++] = b * seg + (t - l / KC);
    }
    return n;
  }
  const long long g0 = (long long)t * KC, g1 = g0 + KC;
  int b = (int)(g0 * B / C);
  while (b + 1 < B && run_lo(C, b + 1, B) <= g0) ++b;
  while (b > 0 && run_lo(C, b, B) > g0) --b;
  int n = 0;
  for (; b < B && run_lo(C, b, B) < g1; ++b) slots[n++] = b * seg + (t - (int)(run_lo(C, b, B) / KC));
  return n;
}

// Sum of the partials at element e (node n, tile row r: e = n * 128 + r)
// over a tile's slot list (from tile_slots), in block order whichever
// kernel adds them (the same rounding).  The loads of a batch of S slots
// (S = 4, 8 or 16, the smallest that holds the list; longer lists take
// several batches) are all issued before the first add, so a sum costs one
// round trip to memory rather than one per four slots; slots past the end of
// the list re-read the last one and are not added.
typedef float f32x8 __attribute__((ext_vector_type(8)));
// fp16 partial values at element e of slot k: 8 (f32x8), 4 (f32x4) or 1 (float)
__device__ __forceinline__ void load_part(const Partials& p, int k, size_t stride, size_t e, f32x8& x, float& sc) {
  const u32x4 h = *reinterpret_cast<const u32x4*>(p.v + k * stride + e);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x2_t v = unpack_f16x2(h[i]);
    x[2 * i] = v[0];
    x[2 * i + 1] = v[1];
  }
  sc = p.sc[k * 4 + (int)(e % kRows) / 32];
}
__device__ __forceinline__ void load_part(const Partials& p, int k, size_t stride, size_t e, f32x4& x, float& sc) {
  const u32x2 h = *reinterpret_cast<const u32x2*>(p.v + k * stride + e);
  const f32x2_t lo = unpack_f16x2(h[0]), hi = unpack_f16x2(h[1]);
  x = f32x4{lo[0], lo[1], hi[0], hi[1]};
  sc = p.sc[k * 4 + (int)(e % kRows) / 32];
}
__device__ __forceinline__ void load_part(const Partials& p, int k, size_t stride, size_t e, float& x, float& sc) {
  x = unpack_f16x2(p.v[k * stride + e])[0];
  sc = p.sc[k * 4 + (int)(e % kRows) / 32];
}
template <typename T, int S>
__device__ __forceinline__ T slot_batches(const Partials& part, const int* slots, int ns, size_t stride, size_t e) {
  T s{};
  for (int i0 = 0; i0 < ns; i0 += S) {
    T x[S];
    float sc[S];
#pragma unroll
    for (int i = 0; i < S; ++i) load_part(part, slots[min(i0 + i, ns - 1)], stride, e, x[i], sc[i]);
#pragma unroll
    for (int i = 0; i < S; ++i)
      if (i0 + i < ns) s += x[i] * sc[i];
  }
  return s;
}
template <typename T>
__device__ __forceinline__ T slot_sum_of(const Partials& part, const int* slots, int ns, size_t stride, size_t e) {
  if (ns <= 4) return slot_batches<T, 4>(part, slots, ns, stride, e);
  if (ns <= 8) return slot_batches<T, 8>(part, slots, ns, stride, e);
  return slot_batches<T, 16>(part, slots, ns, stride, e);
}

// Four blocks per output tile (per gate tile for kSwiGLU): block q takes
// tile rows 64 (q % 2) .. +63 of the nodes n = q / 2 (mod 2); thread item
// (n, 8 consecutive rows), so every partial read is 16 bytes and eight
// lanes read one node's whole 128-byte line.
__global__ __launch_bounds__(256) void linear_reduce_kernel(Partials part, int N, int npad, int K,
                                                            int O, int B, int seg, int epi, void* __restrict__ out,
                                                            int inter) {
  __shared__ int slots[2][256];
  __shared__ int nslots[2];
  const int t = blockIdx.x >> 2, half = blockIdx.x & 1, par = (blockIdx.x >> 1) & 1;
  const int KC = K / 64;
  const int tiles = (O + kRows - 1) / kRows;
  const long long C = (long long)tiles * KC;
  if (threadIdx.x < 2 && (threadIdx.x == 0 || epi == kSwiGLU))
    nslots[threadIdx.x] = tile_slots(C, B, KC, seg, threadIdx.x ? t + inter / kRows : t, slots[threadIdx.x]);
  __syncthreads();
  const size_t stride = (size_t)npad * kRows;  // elements per slot
  const int ns0 = nslots[0], ns1 = epi == kSwiGLU ? nslots[1] : 0;
  for (int item = threadIdx.x; item < (N - par + 1) / 2 * 8; item += 256) {
    const int n = 2 * (item >> 3) + par, r = half * 64 + 8 * (item & 7);
    const size_t e = (size_t)n * kRows + r;
    const int col = t * kRows + r;
    const f32x8 sv = slot_sum_of<f32x8>(part, slots[0], ns0, stride, e);
    if (epi == kSwiGLU) {
      const f32x8 uv = slot_sum_of<f32x8>(part, slots[1], ns1, stride, e);
      uint16_t* o = reinterpret_cast<uint16_t*>(out) + (size_t)n * inter + col;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (col + j < inter) o[j] = (uint16_t)(pack_bf16x2(sv[j] / (1.f + expf(-sv[j])) * uv[j], 0.f) & 0xFFFFu);
      continue;
    }
    const size_t o = (size_t)n * O + col;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (col + j >= O) break;
      if (epi == kStoreF32) reinterpret_cast<float*>(out)[o + j] = sv[j];
      else if (epi == kAddF32) reinterpret_cast<float*>(out)[o + j] += sv[j];
      else reinterpret_cast<uint16_t*>(out)[o + j] = (uint16_t)(pack_bf16x2(sv[j], 0.f) & 0xFFFFu);
    }
  }
}

// Slot-list capacity of the fused epilogues (checked on the host).
constexpr int kMaxTileSlots = 64;
constexpr int kMaxFusedTiles = 64;

// Projection epilogue fused with the next RMSNorm: for row n,
// h[n] += the projection (its partial sums), then out[n] = bf16(h[n] /
// sqrt(mean(h[n]^2) + eps) * w).  One block of 512 threads per row, four
// float4 columns per thread (out_dim <= 8192).
constexpr int kAddNormItems = 4;
__global__ __launch_bounds__(512) void linear_add_rmsnorm_kernel(Partials part, int npad, int K,
                                                                 int O, int B, int seg, float* __restrict__ resid,
                                                                 const uint16_t* __restrict__ w, float eps,
                                                                 uint16_t* __restrict__ out) {
  __shared__ float red[8];
  __shared__ int slots[kMaxFusedTiles][kMaxTileSlots];
  __shared__ int nslots[kMaxFusedTiles];
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int KC = K / 64;
  const int tiles = (O + kRows - 1) / kRows;
  const long long C = (long long)tiles * KC;
  if ((int)threadIdx.x < tiles) nslots[threadIdx.x] = tile_slots(C, B, KC, seg, threadIdx.x, slots[threadIdx.x]);
  __syncthreads();
  const size_t stride = (size_t)npad * kRows;
  float* hrow = resid + (size_t)n * O;
  f32x4 hv[kAddNormItems];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kAddNormItems; ++i) {
    const int c = 4 * (threadIdx.x + 512 * i);
    hv[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (c < O) {
      const int t = c / kRows;
      const f32x4 sv = slot_sum_of<f32x4>(part, slots[t], nslots[t], stride, (size_t)n * kRows + c % kRows);
      hv[i] = *reinterpret_cast<const f32x4*>(hrow + c) + sv;
      *reinterpret_cast<f32x4*>(hrow + c) = hv[i];
    }
  }
#pragma unroll
  for (int i = 0; i < kAddNormItems; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) ss = __builtin_fmaf(hv[i][e], hv[i][e], ss);
  for (int off = 32; off > 0; off >>= 1) ss += shfl_xor_f(ss, off);
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  const float tot = ((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7]));
  const float r = 1.f / sqrtf(tot / (float)O + eps);
#pragma unroll
  for (int i = 0; i < kAddNormItems; ++i) {
    const int c = 4 * (threadIdx.x + 512 * i);
    if (c < O) {
      const u32x2 wv = *reinterpret_cast<const u32x2*>(w + c);
      u32x2 o;
      o[0] = pack_bf16x2(hv[i][0] * r * __uint_as_float(wv[0] << 16), hv[i][1] * r * __uint_as_float(wv[0] & 0xFFFF0000u));
      o[1] = pack_bf16x2(hv[i][2] * r * __uint_as_float(wv[1] << 16), hv[i][3] * r * __uint_as_float(wv[1] & 0xFFFF0000u));
      *reinterpret_cast<u32x2*>(out + (size_t)n * O + c) = o;
    }
  }
}

// Projection epilogue fused with the q/k norms and the rotation: block
// (node n, 16 heads), one wave per head of the fused q/k/v projection.  Lane
// j < D/2 sums the partials of its pair (j, j + D/2) in float32 and then
// proceeds as the rotation kernel: per-head RMSNorm of q and k, rotation at
// position P + depth[n], q to q_out, k and v (rounded to bf16) to cache row
// P + n.
template <int D>
__global__ __launch_bounds__(1024) void linear_qk_norm_rope_kernel(
    Partials part, int npad, int K, int B, int seg, const uint16_t* __restrict__ q_norm,
    const uint16_t* __restrict__ k_norm, float eps, const int32_t* __restrict__ depth, int P,
    const int32_t* __restrict__ P_dev, RopeFreq fr, int Hq, int Hkv, uint16_t* __restrict__ q_out,
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache, long long cap) {
  constexpr int HALF = D / 2;
  static_assert(kRows % D == 0, "a head lies in one tile");
  if (P_dev) P = min(max(*P_dev, 0), P);
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nh = Hq + 2 * Hkv;
  const int hh = blockIdx.y * 16 + wave;
  if (hh >= nh) return;
  __shared__ int slots[16][kMaxTileSlots];
  __shared__ int nslots[16];
  const int KC = K / 64;
  const long long C = (long long)(nh * D / kRows) * KC;
  const size_t stride = (size_t)npad * kRows;
  const int t = hh * D / kRows, r0 = hh * D % kRows;
  if (lane == 0) nslots[wave] = tile_slots(C, B, KC, seg, t, slots[wave]);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const long long row = (long long)P + n;
  const bool act = lane < HALF;
  float a = 0.f, b = 0.f;
  if (act) {
    a = slot_sum_of<float>(part, slots[wave], nslots[wave], stride, (size_t)n * kRows + r0 + lane);
    b = slot_sum_of<float>(part, slots[wave], nslots[wave], stride, (size_t)n * kRows + r0 + lane + HALF);
  }
  if (hh >= Hq + Hkv) {
    uint16_t* dst = v_cache + ((size_t)(hh - Hq - Hkv) * cap + row) * D;
    if (act) {
      dst[lane] = f32_to_bf16_bits(a);
      dst[lane + HALF] = f32_to_bf16_bits(b);
    }
    return;
  }
  float cs = 1.f, sn = 0.f;
  if (act) rope_sincos(P + depth[n], fr.f[lane], sn, cs);
  const bool is_q = hh < Hq;
  norm_rotate(a, b, act, is_q ? q_norm : k_norm, eps, D, lane, cs, sn);
  uint16_t* dst = is_q ? q_out + ((size_t)n * Hq + hh) * D : k_cache + ((size_t)(hh - Hq) * cap + row) * D;
  if (act) {
    dst[lane] = f32_to_bf16_bits(a);
    dst[lane + HALF] = f32_to_bf16_bits(b);
  }
}

struct LinPlan {
  int nb, blocks, seg;
  size_t val_bytes;  // fp16 partial values (the factors follow)
  size_t ws_bytes;
};

Partials partials_in(void* workspace, const LinPlan& p) {
  return Partials{(uint16_t*)workspace, (float*)((uint8_t*)workspace + p.val_bytes)};
}

LinPlan lin_plan(int N, int K, int O) {
  LinPlan p{};
  p.nb = N <= 32 ? 1 : N <= 64 ? 2 : N <= 128 ? 4 : 8;
  const long long C = (long long)((O + kRows - 1) / kRows) * (K / 64);
  const int cus = device_cus() < 256 ? device_cus() : 256;  // the reduce kernel keeps <= 256 slots per tile
  p.blocks = (int)(C < cus ? C : cus);
  const long long run = (C + p.blocks - 1) / p.blocks;
  p.seg = (int)(run / (K / 64)) + 2;  // tiles a run can touch
  p.val_bytes = ((size_t)p.blocks * p.seg * (32 * p.nb) * kRows * sizeof(uint16_t) + 255) / 256 * 256;
  p.ws_bytes = p.val_bytes + (size_t)p.blocks * p.seg * 4 * sizeof(float);
  return p;
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" size_t ooo_linear_packed_bytes(int32_t out_dim, int32_t in_dim) {
  return ooo_lmhead_packed_bytes(out_dim, in_dim, OOO_BF16);
}

extern "C" int ooo_linear_pack(const void* weight, int32_t out_dim, int32_t in_dim, void* packed, size_t packed_bytes,
                               void* stream) {
  return ooo_lmhead_pack(weight, out_dim, in_dim, OOO_BF16, packed, packed_bytes, stream);
}

extern "C" size_t ooo_linear_workspace(int32_t n_rows, int32_t in_dim, int32_t out_dim) {
  if (n_rows < 1 || n_rows > 256 || in_dim < 64 || in_dim % 64 || out_dim < 1) return 0;
  return lin_plan(n_rows, in_dim, out_dim).ws_bytes;
}

// Largest number of stream-K blocks whose runs meet one output tile (the
// length of that tile's slot list).
static int max_tile_slots(int n_rows, int in_dim, int out_dim) {
  const LinPlan p = lin_plan(n_rows, in_dim, out_dim);
  const int KC = in_dim / 64, tiles = (out_dim + kRows - 1) / kRows;
  const long long C = (long long)tiles * KC;
  std::vector<int> count(tiles, 0);
  for (int b = 0; b < p.blocks; ++b) {
    const long long lo = run_lo(C, b, p.blocks), hi = run_lo(C, b + 1, p.blocks);
    if (hi <= lo) continue;
    for (long long t = lo / KC; t <= (hi - 1) / KC; ++t) ++count[t];
  }
  int m = 0;
  for (int c : count) m = c > m ? c : m;
  return m;
}

// Validation and the streaming kernel shared by the entry points; on
// success the partial sums are in the workspace and *plan is set.
static int stream_k(const char* who, const void* x, const void* weight, int32_t n_rows, int32_t in_dim,
                    int32_t out_dim, int32_t weight_layout, void* workspace, size_t ws_bytes, hipStream_t st,
                    LinPlan* plan) {
  OOO_REQUIRE(x && weight, OOO_ERR_INVALID, "%s: null pointer", who);
  OOO_REQUIRE(n_rows >= 1 && in_dim >= 1 && out_dim >= 1, OOO_ERR_INVALID, "%s: sizes must be positive", who);
  OOO_REQUIRE(weight_layout == OOO_W_ROWS || weight_layout == OOO_W_PACKED, OOO_ERR_INVALID,
              "%s: unknown weight layout %d", who, weight_layout);
  OOO_REQUIRE(in_dim % 64 == 0, OOO_ERR_UNSUPPORTED, "%s: in_dim %% 64 != 0", who);
  OOO_REQUIRE(n_rows <= 256, OOO_ERR_UNSUPPORTED, "%s: at most 256 rows", who);
  const LinPlan p = lin_plan(n_rows, in_dim, out_dim);
  OOO_REQUIRE(workspace && ws_bytes >= p.ws_bytes, OOO_ERR_CAPACITY, "%s: workspace of %zu bytes needed (got %zu)",
              who, p.ws_bytes, ws_bytes);
  const uint16_t* X = (const uint16_t*)x;
  const uint16_t* W = (const uint16_t*)weight;
  const Partials part = partials_in(workspace, p);
  const bool pk = weight_layout == OOO_W_PACKED;
#define OOO_LIN_LAUNCH(NBV)                                                                                        \
  do {                                                                                                            \
    if (pk)                                                                                                       \
      linear_bf16_kernel<NBV, true><<<p.blocks, kStreamThreads, 0, st>>>(X, W, n_rows, in_dim, out_dim, p.seg, part);         \
    else                                                                                                          \
      linear_bf16_kernel<NBV, false><<<p.blocks, kStreamThreads, 0, st>>>(X, W, n_rows, in_dim, out_dim, p.seg, part);        \
  } while (0)
  if (p.nb == 1) OOO_LIN_LAUNCH(1);
  else if (p.nb == 2) OOO_LIN_LAUNCH(2);
  else if (p.nb == 4) OOO_LIN_LAUNCH(4);
  else OOO_LIN_LAUNCH(8);
#undef OOO_LIN_LAUNCH
  *plan = p;
  return OOO_OK;
}

extern "C" int ooo_linear(const void* x, const void* weight, int32_t n_rows, int32_t in_dim, int32_t out_dim,
                          int32_t weight_layout, ooo_epilogue epilogue, void* out, void* workspace, size_t ws_bytes,
                          void* stream) {
  OOO_REQUIRE(out, OOO_ERR_INVALID, "ooo_linear: null pointer");
  OOO_REQUIRE(epilogue >= OOO_EPI_STORE_F32 && epilogue <= OOO_EPI_SWIGLU_BF16, OOO_ERR_INVALID,
              "ooo_linear: unknown epilogue %d", (int)epilogue);
  OOO_REQUIRE(epilogue != OOO_EPI_SWIGLU_BF16 || out_dim % 256 == 0, OOO_ERR_UNSUPPORTED,
              "ooo_linear: the SwiGLU epilogue needs out_dim %% 256 == 0 (gate and up halves of whole tiles)");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  LinPlan p{};
  const int rc = stream_k("ooo_linear", x, weight, n_rows, in_dim, out_dim, weight_layout, workspace, ws_bytes, st, &p);
  if (rc != OOO_OK) return rc;
  const Partials part = partials_in(workspace, p);
  const int tiles = (out_dim + kRows - 1) / kRows;
  const int rgrid = 4 * (epilogue == OOO_EPI_SWIGLU_BF16 ? tiles / 2 : tiles);
  linear_reduce_kernel<<<rgrid, 256, 0, st>>>(part, n_rows, 32 * p.nb, in_dim, out_dim, p.blocks, p.seg, (int)epilogue,
                                              out, out_dim / 2);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_linear: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_linear_add_rmsnorm(const void* x, const void* weight, int32_t n_rows, int32_t in_dim,
                                      int32_t out_dim, int32_t weight_layout, float* residual,
                                      const void* norm_weight, float eps, void* normed_out, void* workspace,
                                      size_t ws_bytes, void* stream) {
  OOO_REQUIRE(residual && norm_weight && normed_out, OOO_ERR_INVALID, "ooo_linear_add_rmsnorm: null pointer");
  OOO_REQUIRE(eps >= 0.f, OOO_ERR_INVALID, "ooo_linear_add_rmsnorm: eps must be >= 0");
  OOO_REQUIRE(out_dim % 4 == 0 && out_dim <= 512 * 4 * kAddNormItems, OOO_ERR_UNSUPPORTED,
              "ooo_linear_add_rmsnorm: out_dim %d must be a multiple of 4 and at most %d", out_dim,
              512 * 4 * kAddNormItems);
  OOO_REQUIRE(n_rows < 1 || in_dim < 64 || in_dim % 64 || n_rows > 256 ||
                  max_tile_slots(n_rows, in_dim, out_dim) <= kMaxTileSlots,
              OOO_ERR_UNSUPPORTED, "ooo_linear_add_rmsnorm: more than %d partial slots per tile at this shape",
              kMaxTileSlots);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  LinPlan p{};
  const int rc = stream_k("ooo_linear_add_rmsnorm", x, weight, n_rows, in_dim, out_dim, weight_layout, workspace,
                          ws_bytes, st, &p);
  if (rc != OOO_OK) return rc;
  linear_add_rmsnorm_kernel<<<n_rows, 512, 0, st>>>(partials_in(workspace, p), 32 * p.nb, in_dim, out_dim, p.blocks,
                                                     p.seg, residual, (const uint16_t*)norm_weight, eps,
                                                     (uint16_t*)normed_out);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_linear_add_rmsnorm: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_linear_qk_norm_rope(const void* x, const void* weight, int32_t n_rows, int32_t in_dim,
                                       int32_t weight_layout, const void* q_norm, const void* k_norm, float eps,
                                       const int32_t* depth, int32_t prefix_len, const int32_t* prefix_len_dev,
                                       double rope_theta, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                       void* q_out, void* k_cache, void* v_cache, int64_t cap, void* workspace,
                                       size_t ws_bytes, void* stream) {
  OOO_REQUIRE(depth && q_out && k_cache && v_cache, OOO_ERR_INVALID, "ooo_linear_qk_norm_rope: null pointer");
  OOO_REQUIRE(n_q_heads >= 1 && n_kv_heads >= 1 && prefix_len >= 0, OOO_ERR_INVALID,
              "ooo_linear_qk_norm_rope: sizes must be positive");
  OOO_REQUIRE((int64_t)prefix_len + n_rows <= cap, OOO_ERR_INVALID,
              "ooo_linear_qk_norm_rope: prefix_len + n_rows (%lld) exceeds cap (%lld)", (long long)prefix_len + n_rows,
              (long long)cap);
  OOO_REQUIRE(rope_theta > 0.0 && eps >= 0.f, OOO_ERR_INVALID, "ooo_linear_qk_norm_rope: rope_theta must be > 0");
  OOO_REQUIRE(head_dim == 64 || head_dim == 128, OOO_ERR_UNSUPPORTED,
              "ooo_linear_qk_norm_rope: head_dim %d not supported (64 or 128)", head_dim);
  const int nh = n_q_heads + 2 * n_kv_heads;
  OOO_REQUIRE((int64_t)nh * head_dim % kRows == 0, OOO_ERR_UNSUPPORTED,
              "ooo_linear_qk_norm_rope: (n_q_heads + 2 n_kv_heads) * head_dim must be a multiple of %d", kRows);
  OOO_REQUIRE(n_rows < 1 || in_dim < 64 || in_dim % 64 || n_rows > 256 ||
                  max_tile_slots(n_rows, in_dim, nh * head_dim) <= kMaxTileSlots,
              OOO_ERR_UNSUPPORTED, "ooo_linear_qk_norm_rope: more than %d partial slots per tile at this shape",
              kMaxTileSlots);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  LinPlan p{};
  const int rc = stream_k("ooo_linear_qk_norm_rope", x, weight, n_rows, in_dim, nh * head_dim, weight_layout,
                          workspace, ws_bytes, st, &p);
  if (rc != OOO_OK) return rc;
  const RopeFreq fr = rope_freq(rope_theta, head_dim);
  const dim3 grid(n_rows, (nh + 15) / 16);
  const Partials part = partials_in(workspace, p);
  if (head_dim == 128)
    linear_qk_norm_rope_kernel<128><<<grid, 1024, 0, st>>>(part, 32 * p.nb, in_dim, p.blocks, p.seg,
                                                            (const uint16_t*)q_norm, (const uint16_t*)k_norm, eps, depth,
                                                            prefix_len, prefix_len_dev, fr, n_q_heads, n_kv_heads,
                                                            (uint16_t*)q_out, (uint16_t*)k_cache, (uint16_t*)v_cache,
                                                            cap);
  else
    linear_qk_norm_rope_kernel<64><<<grid, 1024, 0, st>>>(part, 32 * p.nb, in_dim, p.blocks, p.seg,
                                                           (const uint16_t*)q_norm, (const uint16_t*)k_norm, eps, depth,
                                                           prefix_len, prefix_len_dev, fr, n_q_heads, n_kv_heads,
                                                           (uint16_t*)q_out, (uint16_t*)k_cache, (uint16_t*)v_cache,
                                                           cap);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_linear_qk_norm_rope: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
