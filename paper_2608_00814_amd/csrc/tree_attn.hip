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
//    A split is a fixed-length run of tiles, so the key ranges a row's
//    partial sums cover (and its rounding) do not depend on the row block:
//    for a given key layout a node's output is bitwise the same in tries of
//    any size that get the same split count (the count depends on the trie
//    size only where the CUs limit it).
//  * Scores are computed transposed, S^T = K Q^T, and the output as
//    O^T = V^T P^T.  With the A-operand rows of K permuted (bits 2 and 3 of
//    the row index swapped) every lane ends up holding one query row: its
//    softmax state, its probabilities (already in B-operand order for the
//    second product) and 16 of its output columns, so the online softmax
//    needs one cross-lane exchange per tile and no LDS round trip.
//  * K and V tiles stream into a 4-stage LDS ring by DMA (global_load_lds);
//    the V^T operand is read from the row-major V tile with transposing LDS
//    reads (ds_read_b64_tr_b16).
//  * head_dim 128: two waves per 32-row group, each taking one 32-key half
//    of every tile (two waves per SIMD); head_dim 64: one wave per row group
//    with a hand-pipelined tile loop.
//  * Splits write fp16 partials (normalised O times a power of two, plus
//    the split's log2 weight and the power's exponent, 8 bytes per row)
//    that a second kernel combines, loading exactly the splits there are;
//    with one split the kernel writes O directly.
//  * Launch order is XCD-aware: consecutive work items (same KV head and
//    row block, neighbouring splits) go to blocks that share blockIdx % 8,
//    so one head's K/V stream stays in one XCD's L2.
#include <math.h>
#include <stdlib.h>

#include <mutex>
#include <type_traits>

#include "device_common.h"
#include "ooo_internal.h"

namespace ooo {
namespace {

constexpr int kTile = 64;         // keys per tile
constexpr int kMaxMaskWords = 16;  // ancestor-mask words per node (up to 1024 nodes)

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
  uint32_t* part_o;  // fp16 normalised partial outputs (fragment order)
  float* part_ml;    // per partial row: log2 of the split's weight, exponent of its scale
  int splits, row_blocks, Mpad, tiles_prefix, tiles_total;
  int tps;           // key tiles per split (split s takes tiles [s tps, (s + 1) tps))
  const int* P_dev;  // null, or the prefix length in device memory (P bounds it)
};

// swap bits 2 and 3: the K row a lane loads so that S^T lands with eight
// consecutive keys per lane and k-step
__device__ __forceinline__ int sigma(int c) { return (c & ~0xC) | ((c & 4) << 1) | ((c & 8) >> 1); }

typedef short i16x4 __attribute__((ext_vector_type(4)));
// Kernel-local lambdas must be inlined: an outlined call would take its
// captures through memory and lose their wave-uniformity (the DMA needs
// scalar operands).
#define OOO_INLINE __attribute__((always_inline))

// LDS DMA of 16 bytes per lane from base + voff (base wave-uniform, voff
// per lane); lane l's bytes land at LDS byte address lds + 16*l (lds
// wave-uniform).  Issued through inline asm so the compiler does not track
// it: it would otherwise make LDS reads of other ring stages wait for every
// DMA in flight.  Kernels wait for their DMA explicitly (vmcnt, then a
// barrier).  M0 holds the LDS base; nothing else in these kernels uses M0.
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(voff), "s"(base)
               : "memory", "m0");
}

// Same with the non-temporal (streaming) cache policy, for the K/V tiles:
// each head's K/V stream is read once per row block, and keeping it from
// displacing the rest of the L2 (the queries every split re-reads, the
// partials) measured 16.6 -> 15.5 us per call at the Qwen3-8B shape.
__device__ __forceinline__ void dma16_nt(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(lds), "v"(voff), "s"(base)
               : "memory", "m0");
}

// Same for 4 bytes per lane (lane l's dword lands at lds + 4*l).
__device__ __forceinline__ void dma4(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(voff), "s"(base)
               : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// max of three floats without the NaN canonicalisation fmaxf implies
// (scores are finite or -inf)
__device__ __forceinline__ float max3f(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// LDS ring geometry for one head_dim.  A tile is 64 rows of K and 64 rows of
// V, each row D bf16 values = D/8 16-byte chunks, stored row-major with the
// chunks of a row permuted (swz below).  One 1 KiB DMA instruction copies
// whole contiguous rows (coalesced in global memory).  Every stage of every
// matrix is its own __shared__ array, so the compiler can tell that a DMA
// into one stage does not alias reads of another and adds no waits of its
// own; the kernel waits explicitly (vmcnt, then a barrier).
template <int D>
struct Ring {
  static constexpr int CH = D / 8;            // chunks per row
  static constexpr int ROWB = 2 * D;          // bytes per row
  static constexpr int MAT = kTile * ROWB;    // bytes of one K or V tile
  static constexpr int NS = 4;                // stages
  static constexpr int DMA_MAT = MAT / 1024;  // DMA instructions per matrix
  static constexpr int RPI = 1024 / ROWB;     // rows per DMA instruction
  static constexpr int GPL = D / 8;           // float4 groups of O^T per lane
  // Physical chunk of logical chunk c in row r.  For D = 128 the two 2-bit
  // halves of r % 16 are swapped and XORed in: the K fragment reads (16
  // lanes, 16 different rows, one chunk) and the V transpose reads (32
  // lanes, 4 consecutive rows x 4 consecutive chunks) both hit distinct banks.
  static __device__ __forceinline__ int swz(int r, int c) {
    if (D == 128) return c ^ (((r & 3) << 2) | ((r >> 2) & 3));
    return c ^ (r % CH);
  }
};

// wait until at most `ahead` tiles of `per` DMA instructions are pending
template <int PER, int MAXA>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if (MAXA >= 2 && ahead >= 2) wait_vmcnt<(MAXA >= 2 ? 2 * PER : 0)>();
  else if (ahead == 1) wait_vmcnt<PER>();
  else wait_vmcnt<0>();
}

// Work of one block: RG row groups of 32 query rows.  Without SPLIT one
// wave per row group reads all 64 keys of every tile; with SPLIT two waves
// share a row group, each taking one 32-key half of every tile, so that two
// waves sit on each SIMD and the matrix-core work of one overlaps the vector
// work of the other; the halves merge their (max, sum, O) through LDS at the
// end.  Within a wave the loop is software-pipelined: while the matrix cores
// compute the scores of tile i+1 (S^T = K Q^T), the vector units turn the
// scores of tile i into probabilities; the P V product of tile i overlaps the
// row max of tile i+1.  LDS reads are issued one phase ahead of their use.
// Every wave issues its share of each tile's DMA.
template <int D, int RG, bool SPLIT>
__global__ __launch_bounds__(64 * RG * (SPLIT ? 2 : 1)) void tree_attn_bf16_kernel(AttnArgs a) {
  using R = Ring<D>;
  constexpr int NW = RG * (SPLIT ? 2 : 1);  // waves
  constexpr int NH = SPLIT ? 1 : 2;         // 32-key halves per wave and tile
  constexpr int BM = 32 * RG;               // query rows per block
  constexpr int PM = R::DMA_MAT / NW;       // DMA instructions per wave per matrix
  constexpr int PER = 2 * PM;               // ... per tile
  static_assert(R::DMA_MAT % NW == 0, "DMA split");
  static_assert(2 * PER <= 63, "vmcnt range");
  static_assert(R::GPL % 4 == 0, "merge layout");
  __shared__ __attribute__((aligned(1024))) uint8_t k0[R::MAT], k1[R::MAT], k2[R::MAT], k3[R::MAT];
  __shared__ __attribute__((aligned(1024))) uint8_t v0[R::MAT], v1[R::MAT], v2[R::MAT], v3[R::MAT];
  // ancestor-mask words of the block's rows (a wave reads only its own rows)
  __shared__ uint64_t mwords[RG * 32 * kMaxMaskWords];
  uint8_t* const kst[R::NS] = {k0, k1, k2, k3};
  uint8_t* const vst[R::NS] = {v0, v1, v2, v3};

  const int total = a.Hkv * a.row_blocks * a.splits;
  int w = blockIdx.x;
  if (total % 8 == 0) w = (w % 8) * (total / 8) + w / 8;
  const int s = w % a.splits;
  w /= a.splits;
  const int rb = w % a.row_blocks;
  const int g = w / a.row_blocks;
  // The prefix length is the launch value or, for replays of one captured
  // step at a growing prefix, the value in device memory (clamped to the
  // launch value, which the plan and the validation used).
  const int P = a.P_dev ? __builtin_amdgcn_readfirstlane(min(max(*a.P_dev, 0), a.P)) : a.P;
  const int tiles_prefix = (P + kTile - 1) / kTile;
  const int tiles_total = tiles_prefix + (a.N + kTile - 1) / kTile;
  // Fixed-length runs of tiles, the length set by the actual prefix (with
  // a device prefix the plan's split count is spread over the tiles the
  // prefix has; with the launch value this is the plan's length), so a
  // row's key ranges and its rounding do not depend on the row block.  The
  // last splits can be empty when there are fewer tiles than splits
  // (handled below).
  const int tps = a.P_dev ? (tiles_total + a.splits - 1) / a.splits : a.tps;
  const int t_begin = s * tps;
  const int t_end = min(t_begin + tps, tiles_total);
  const int ntiles = t_end - t_begin;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int rg = wave % RG, kh0 = SPLIT ? wave / RG : 0;
  const int c = lane & 31, u = lane >> 5;
  uint64_t* const mrow = mwords + (rg * 32 + c) * kMaxMaskWords;
  const int row = rb * BM + rg * 32 + c;
  const bool row_ok = row < a.M;
  const int rr = row_ok ? row : a.M - 1;
  const int node = rr / a.G;
  const int head = g * a.G + (rr - node * a.G);
  const uint16_t* const kg = a.k + (size_t)g * a.cap * D;
  const uint16_t* const vg = a.v + (size_t)g * a.cap * D;

  if (ntiles <= 0) {
    // Empty split (only with a device prefix shorter than the plan's; then
    // splits > 1): a partial with no allowed key, zero weight in the merge.
    if (kh0 != 0 || !row_ok) return;
    const size_t blk = ((size_t)s * a.Hkv + g) * (a.Mpad / 32) + (row >> 5);
    u32x4* po = reinterpret_cast<u32x4*>(a.part_o) + blk * (R::GPL / 2) * 64 + lane;
#pragma unroll
    for (int k = 0; k < R::GPL / 2; ++k) po[k * 64] = u32x4{0u, 0u, 0u, 0u};
    if (u == 0)
      *reinterpret_cast<f32x2_t*>(a.part_ml + (((size_t)s * a.Hkv + g) * a.Mpad + row) * 2) =
          f32x2_t{-INFINITY, 0.f};
    return;
  }

  // Q^T fragments (B operand of S^T = K Q^T): row c, k = 16dk + 8u .. +8.
  // The key-split kernel stages Q through LDS instead (below).
  bf16x8 qf[D / 16];
  if constexpr (!SPLIT) {
    const uint16_t* qrow = a.q + ((size_t)node * a.Hq + head) * D;
#pragma unroll
    for (int dk = 0; dk < D / 16; ++dk) qf[dk] = as_bf16x8(ld16(qrow + 16 * dk + 8 * u));
  }

  auto tile_rows = [&](int t, int& row0, int& limit) OOO_INLINE {
    if (t < tiles_prefix) {
      row0 = t * kTile;
      limit = P;
    } else {
      row0 = P + (t - tiles_prefix) * kTile;
      limit = P + a.N;
    }
  };
  // DMA instruction j of a matrix copies rows RPI*j .. +RPI: lane = (row
  // within the instruction, physical chunk), so it reads the logical chunk
  // swz(r, physical) of row r.  Interior tiles use the per-lane byte offsets
  // below from a uniform tile base; a tile that crosses the end of its
  // region clamps rows past it to the last valid row (masked keys, zero
  // probability).
  uint32_t dvoff[PM];
#pragma unroll
  for (int i = 0; i < PM; ++i) {
    const int r = (i * NW + wave) * R::RPI + lane / R::CH;
    dvoff[i] = r * R::ROWB + R::swz(r, lane % R::CH) * 16;
  }
  auto issue = [&](int t, auto stage_c) OOO_INLINE {
    constexpr int ST = decltype(stage_c)::value;
    int row0, limit;
    tile_rows(t, row0, limit);
    const uint16_t* kb = kg + (size_t)row0 * D;
    const uint16_t* vb = vg + (size_t)row0 * D;
    const uint32_t kl = lds_addr(kst[ST]) + wave_u * 1024, vl = lds_addr(vst[ST]) + wave_u * 1024;
    if (row0 + kTile <= limit) {
#pragma unroll
      for (int i = 0; i < PM; ++i) dma16_nt(kb, dvoff[i], kl + i * NW * 1024);
#pragma unroll
      for (int i = 0; i < PM; ++i) dma16_nt(vb, dvoff[i], vl + i * NW * 1024);
    } else {
      uint32_t vo[PM];
#pragma unroll
      for (int i = 0; i < PM; ++i) {
        const int r = (i * NW + wave) * R::RPI + lane / R::CH;
        const int rc = min(r, limit - 1 - row0);
        vo[i] = rc * R::ROWB + R::swz(r, lane % R::CH) * 16;
      }
#pragma unroll
      for (int i = 0; i < PM; ++i) dma16_nt(kb, vo[i], kl + i * NW * 1024);
#pragma unroll
      for (int i = 0; i < PM; ++i) dma16_nt(vb, vo[i], vl + i * NW * 1024);
    }
  };
  // Every tile issues its PM K instructions before its PM V instructions,
  // so waiting until PM are pending leaves only the tile's V in flight.

  // The mask words go through LDS so that no global load is pending inside
  // the tile loop, where a wait for it would also wait for the tile DMA.
  if constexpr (!SPLIT) {
    for (int wd = u; wd < a.W; wd += 2) mrow[wd] = a.mask[(size_t)node * a.W + wd];
  } else {
    // Key-split kernel: Q and the mask words arrive by DMA as well, so the
    // kernel has no compiler-tracked load at all (the compiler would wait
    // for one with vmcnt(0), which also waits for every tile in flight).
    // Q rows of the block, row-major with the K chunk permutation, go to
    // ring stage 3 (rows 0..63 in k3, 64..127 in v3): tile 3 is not
    // requested before every wave has read its fragments.  Mask words go
    // to mwords as [row][W] (dword DMA, 64 dwords per instruction).
    const auto row_src = [&](int r) OOO_INLINE {
      const int rq = min(rb * BM + r, a.M - 1);
      return rq / a.G;
    };
    for (int j = wave_u; j < BM / R::RPI; j += NW) {
      const int r = j * R::RPI + lane / R::CH;
      const int rq = min(rb * BM + r, a.M - 1);
      const int nd = rq / a.G;
      const uint32_t off = (uint32_t)((nd * a.Hq + g * a.G + (rq - nd * a.G)) * D) * 2u +
                           (uint32_t)R::swz(r, lane % R::CH) * 16u;
      const uint32_t dst = j * R::RPI < 64 ? lds_addr(k3) + j * 1024 : lds_addr(v3) + (j - 64 / R::RPI) * 1024;
      dma16(a.q, off, dst);
    }
    const int nmask = BM * 2 * a.W / 64;  // dword instructions
    for (int j = wave_u; j < nmask; j += NW) {
      const int e = j * 64 + lane;
      const int r = e / (2 * a.W), k = e - r * (2 * a.W);
      dma4(a.mask, (uint32_t)(row_src(r) * 2 * a.W + k) * 4u, lds_addr(mwords) + j * 256);
    }
  }

  // Only the first tile is requested up front: when every block asks for
  // several tiles at once, each block's first tile lands late.
  issue(t_begin, std::integral_constant<int, 0>{});

  // Per-lane LDS byte offsets (loop invariant).  K fragment (half kh,
  // k-step dk): logical chunk 2dk+u of row sigma(c) + 32kh (the physical
  // chunk only depends on the row mod 16).  V^T transpose-read source
  // (column block dt, key step ks, half h): row 16ks + 4h + 8(g16/2) + li/4,
  // columns 32dt + 16(g16%2) + 4(li%4) .. +3.
  const int krow = sigma(c);
  uint32_t koff[D / 16];
#pragma unroll
  for (int dk = 0; dk < D / 16; ++dk)
    koff[dk] = (krow + 32 * kh0) * R::ROWB + (R::swz(krow, 2 * dk + u) << 4);
  const int g16 = lane >> 4, li = lane & 15;
  uint32_t voff[D / 32][2];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int vr = 4 * h + 8 * (g16 >> 1) + (li >> 2);  // key row within a 16-row block
      const int col = 32 * dt + 16 * (g16 & 1) + 4 * (li & 3);
      voff[dt][h] = (vr + 32 * kh0) * R::ROWB + (R::swz(vr, col >> 3) << 4) + (col & 7) * 2;
    }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // K fragments of k-steps 4b .. 4b+3 for the wave's halves
  auto kread = [&](auto stage_c, int b, bf16x8 (&kf)[NH][4]) OOO_INLINE {
    constexpr int ST = decltype(stage_c)::value;
    const uint8_t* Ks = kst[ST];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int hf = 0; hf < NH; ++hf)
        kf[hf][j] = as_bf16x8(*reinterpret_cast<const u32x4*>(Ks + koff[4 * b + j] + 32 * hf * R::ROWB));
  };
  auto qk_mfma = [&](int b, const bf16x8 (&kf)[NH][4], f32x16 (&acc)[NH]) OOO_INLINE {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int hf = 0; hf < NH; ++hf) acc[hf] = mfma32(kf[hf][j], qf[4 * b + j], acc[hf]);
  };
  // V^T fragments of local key step ks (16 keys of the wave's range)
  auto vread = [&](auto stage_c, int ks, bf16x8 (&vv)[D / 32]) OOO_INLINE {
    constexpr int ST = decltype(stage_c)::value;
    const uint8_t* Vs = vst[ST];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
      u32x2 lohi[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint8_t* p = Vs + voff[dt][h] + ks * 16 * R::ROWB;
        lohi[h] = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((i16x4 __attribute__((address_space(3)))*)OOO_LDS(p)));
      }
      vv[dt] = as_bf16x8(u32x4{lohi[0][0], lohi[0][1], lohi[1][0], lohi[1][1]});
    }
  };
  auto pv_mfma = [&](const bf16x8 (&vv)[D / 32], const bf16x8& p) OOO_INLINE {
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = mfma32(vv[dt], p, oacc[dt]);
  };
  // probabilities of one 32-key half in B-operand order; returns their sum
  auto probs_half = [&](const f32x16& acc, float m_use, bf16x8& p0, bf16x8& p1) OOO_INLINE {
    float ps[4] = {0.f, 0.f, 0.f, 0.f};  // four independent sums: short dependency chains
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      float p[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = __builtin_amdgcn_exp2f(fmaf(acc[8 * k2 + e], a.scale_log2e, -m_use));
        ps[e % 4] += p[e];
      }
      u32x4 pk;
#pragma unroll
      for (int e = 0; e < 4; ++e) pk[e] = pack_bf16x2(p[2 * e], p[2 * e + 1]);
      (k2 == 0 ? p0 : p1) = as_bf16x8(pk);
    }
    return (ps[0] + ps[1]) + (ps[2] + ps[3]);
  };
  // Mask tile t's scores (tree tiles and ragged tails only).  Lane value j
  // of half hf is key 32(kh0+hf) + 16*(j/8) + 8u + j%8 of the tile.
  auto apply_mask = [&](int t, f32x16 (&acc)[NH]) OOO_INLINE {
    int row0, limit;
    tile_rows(t, row0, limit);
    const bool tree = t >= tiles_prefix;
    if (tree || row0 + kTile > limit) {
      const uint64_t mw =
          !tree ? ~0ull : SPLIT ? mwords[(rg * 32 + c) * a.W + (t - tiles_prefix)] : mrow[t - tiles_prefix];
      // A lane's values are two runs of 8 consecutive keys: each run's 8
      // mask bits come from one shift.  (Testing a precomputed bit per key
      // kept 48 registers live through the whole tile loop: 249 -> 200
      // VGPRs for the key-split kernel, 16.40 -> 16.14 us per call at the
      // Qwen3-8B shape.)
      const int rem = limit - row0;  // keys of the tile inside the region
#pragma unroll
      for (int hf = 0; hf < NH; ++hf)
#pragma unroll
        for (int g8 = 0; g8 < 2; ++g8) {
          const int base = 32 * (kh0 + hf) + 16 * g8 + 8 * u;
          const int inside = rem - base;
          uint32_t bits = (uint32_t)(mw >> base) & 0xffu;
          bits &= inside >= 8 ? 0xffu : inside <= 0 ? 0u : (1u << inside) - 1u;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (!((bits >> e) & 1u)) acc[hf][8 * g8 + e] = -INFINITY;
        }
    }
  };
  // row max of a tile's scores over the wave's keys, in log2 units
  auto row_max = [&](const f32x16 (&acc)[NH]) OOO_INLINE {
    float mh[NH];
#pragma unroll
    for (int hf = 0; hf < NH; ++hf) {  // two interleaved chains
      float m0 = max3f(acc[hf][0], acc[hf][1], acc[hf][2]);
      float m1 = max3f(acc[hf][8], acc[hf][9], acc[hf][10]);
      m0 = max3f(m0, acc[hf][3], acc[hf][4]);
      m1 = max3f(m1, acc[hf][11], acc[hf][12]);
      m0 = max3f(m0, acc[hf][5], acc[hf][6]);
      m1 = max3f(m1, acc[hf][13], acc[hf][14]);
      mh[hf] = max3f(max3f(m0, acc[hf][7], m1), acc[hf][15], -INFINITY);
    }
    const float mx = NH == 2 ? max3f(mh[0], mh[NH - 1], -INFINITY) : mh[0];
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    return max3f(__uint_as_float(sw[0]), __uint_as_float(sw[1]), -INFINITY) * a.scale_log2e;
  };
  // Lazy rescaling: the reference max m_run moves only when some row of the
  // wave grows by more than 2^8, so probabilities stay <= 256 (fine for fp32
  // sums and bf16 operands) and O, l are rescaled rarely.
  auto rescale = [&](float mx) OOO_INLINE {
    if (__any(mx > m_run + 8.f)) {
      const float m_new = __builtin_fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - (m_new == -INFINITY ? 0.f : m_new));
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;
      m_run = m_new;
    }
  };

  if constexpr (SPLIT) {
    // Two waves per SIMD, one per key half of the same rows, half a tile
    // apart: wave A (kh0 = 0) runs scores, softmax and P V of tile i between
    // barriers i and i+1; wave B runs P V of tile i-1, then scores and
    // softmax of tile i.  So while one wave is in its softmax (vector
    // units) the other issues matrix-core work.  Because B reads V of tile
    // i-1 after barrier i, the ring runs two tiles ahead: barrier i is
    // followed by the DMA of tile i+2 into the stage of tile i-2.
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    // Tile 0 landed (the compiler does not track the DMA, so the barrier
    // alone would not wait for it); the mask words in LDS are visible.  Tile
    // 1 is requested only now: with every block asking for tiles 0 and 1 at
    // once, each block's tile 0 lands later (15.57 -> 15.41 us per call at
    // the Qwen3-8B shape, graphs of 36 calls).
    // Only K of tile 0 (and Q, the mask words) must have landed: V of tile
    // 0 is first read after barrier 1, whose wait covers it (with a single
    // tile it is read before any other wait, so then wait for it too).
    if (ntiles > 1) wait_vmcnt<PM>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (ntiles > 1) issue(t_begin + 1, I1{});
    {
      const int rq = rg * 32 + c;
      const uint8_t* qs = (rg < 2 ? k3 : v3) + (rq % 64) * R::ROWB;
#pragma unroll
      for (int dk = 0; dk < D / 16; ++dk)
        qf[dk] = as_bf16x8(*reinterpret_cast<const u32x4*>(qs + (R::swz(rq, 2 * dk + u) << 4)));
    }
    if (ntiles > 2) issue(t_begin + 2, I2{});
    // Both waves of a pair run each tile as one matrix block (P V of the
    // previous tile, then the scores of this one) and one vector block (the
    // softmax): wave A (kh0 = 0) matrix block first, wave B (kh0 = 1)
    // vector block first, so that on their SIMD the matrix cores work for
    // one wave while the vector units work for the other.  A keeps the
    // probabilities of the previous tile, B its scores.
    auto pv_tile = [&](auto stage_c, const bf16x8 (&pf)[2]) OOO_INLINE {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bf16x8 vv[D / 32];
        vread(stage_c, ks, vv);
        pv_mfma(vv, pf[ks]);
      }
    };
    bf16x8 pf_hold[2];   // A: probabilities of the previous tile
    f32x16 sc_hold[1];   // B: scores of the previous tile
    auto softmax_tile = [&](int t, f32x16 (&sc)[1]) OOO_INLINE {
      apply_mask(t, sc);
      rescale(row_max(sc));
      l_run += probs_half(sc[0], m_run == -INFINITY ? 0.f : m_run, pf_hold[0], pf_hold[1]);
    };
    auto body = [&](auto role_c, int i, auto st_c) OOO_INLINE {
      constexpr bool B = decltype(role_c)::value;
      constexpr int ST = decltype(st_c)::value;
      if (i > 0) {
        wait_tiles<PER, 1>(min(1, ntiles - 1 - i));  // this wave's share of tile i landed
        wg_barrier();                                // ... and every other wave's
        if constexpr (B) softmax_tile(t_begin + i - 1, sc_hold);
        __builtin_amdgcn_sched_barrier(0);
        pv_tile(std::integral_constant<int, (ST + 3) % 4>{}, pf_hold);
      }
      f32x16 sc[1] = {f32x16{}};
      bf16x8 kf[1][4];
#pragma unroll
      for (int b = 0; b < D / 64; ++b) {
        kread(st_c, b, kf);
        qk_mfma(b, kf, sc);
      }
      // The DMA of tile i+2 (into the stage tile i-2 used, free since this
      // tile's barrier) is issued once the matrix block is under way.
      if (i > 0 && i + 2 < ntiles) issue(t_begin + i + 2, std::integral_constant<int, (ST + 2) % 4>{});
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (!B) softmax_tile(t_begin + i, sc);
      else sc_hold[0] = sc[0];
      if (i == ntiles - 1) {  // the last tile's P V
        if constexpr (B) softmax_tile(t_begin + i, sc_hold);
        pv_tile(st_c, pf_hold);
      }
    };
    auto run = [&](auto role_c) OOO_INLINE {
      int i = 0;
      for (; i + 4 <= ntiles; i += 4) {
        body(role_c, i, I0{});
        body(role_c, i + 1, I1{});
        body(role_c, i + 2, I2{});
        body(role_c, i + 3, I3{});
      }
      if (i < ntiles) body(role_c, i, I0{});
      if (i + 1 < ntiles) body(role_c, i + 1, I1{});
      if (i + 2 < ntiles) body(role_c, i + 2, I2{});
    };
    if (__builtin_amdgcn_readfirstlane(kh0) == 0) run(std::false_type{});
    else run(std::true_type{});
  } else {
  // prologue: scores, mask and max of the first tile
    f32x16 sa_buf[NH], sb_buf[NH];
    wait_vmcnt<0>();
    wg_barrier();
    if (ntiles > 1) issue(t_begin + 1, std::integral_constant<int, 1>{});
    if (ntiles > 2) issue(t_begin + 2, std::integral_constant<int, 2>{});
    {
      bf16x8 kf[NH][4];
#pragma unroll
      for (int hf = 0; hf < NH; ++hf) sa_buf[hf] = f32x16{};
#pragma unroll
      for (int b = 0; b < D / 64; ++b) {
        kread(std::integral_constant<int, 0>{}, b, kf);
        qk_mfma(b, kf, sa_buf);
      }
    }
    apply_mask(t_begin, sa_buf);
    rescale(row_max(sa_buf));

    // One pipeline step: tile i is in stage SA with its scores in scur, tile
    // i+1 (if NEXT) in stage SB, its scores go to snxt; tile i+3 is issued
    // into SD, the stage tile i-1 used.  The row max of tile i+1 is taken
    // before masking; a masked tile (tree tiles, ragged tails) takes it again
    // after the mask.  Phases are separated by scheduling barriers.
    auto step = [&](int i, auto sa, auto sb, auto sd, auto next_c, f32x16 (&scur)[NH], f32x16 (&snxt)[NH]) OOO_INLINE {
      constexpr bool NEXT = decltype(next_c)::value;
      if (NEXT) {
        wait_tiles<PER, 1>(min(1, ntiles - 2 - i));  // this wave's share of tile i+1 landed
        wg_barrier();                                // ... and every other wave's
        if (i + 3 < ntiles) issue(t_begin + i + 3, sd);
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run;
      bf16x8 pf[2 * NH];
      bf16x8 vv0[D / 32], vv1[D / 32];
      if (NEXT) {
        bf16x8 kf[NH][4];
        __builtin_amdgcn_sched_barrier(0);
        kread(sb, 0, kf);
        vread(sa, 0, vv0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int hf = 0; hf < NH; ++hf) snxt[hf] = f32x16{};
        qk_mfma(0, kf, snxt);
        float ps = probs_half(scur[0], m_use, pf[0], pf[1]);
        if (D / 64 > 1) kread(sb, 1, kf);
        __builtin_amdgcn_sched_barrier(0);
        if (D / 64 > 1) qk_mfma(1, kf, snxt);
        if (NH == 2) ps += probs_half(scur[NH - 1], m_use, pf[2 * NH - 2], pf[2 * NH - 1]);
        vread(sa, 1, vv1);
        l_run += ps;
        __builtin_amdgcn_sched_barrier(0);
        pv_mfma(vv0, pf[0]);
        if (NH == 2) vread(sa, 2, vv0);
        __builtin_amdgcn_sched_barrier(0);
        pv_mfma(vv1, pf[1]);
        if (NH == 2) vread(sa, 3, vv1);
        float mx = row_max(snxt);
        __builtin_amdgcn_sched_barrier(0);
        if (NH == 2) {
          pv_mfma(vv0, pf[2 * NH - 2]);
          pv_mfma(vv1, pf[2 * NH - 1]);
        }
        __builtin_amdgcn_sched_barrier(0);
        int row0, limit;
        tile_rows(t_begin + i + 1, row0, limit);
        if (t_begin + i + 1 >= tiles_prefix || row0 + kTile > limit) {
          apply_mask(t_begin + i + 1, snxt);
          mx = row_max(snxt);
        }
        rescale(mx);
      } else {
        float ps = 0.f;
#pragma unroll
        for (int hf = 0; hf < NH; ++hf) ps += probs_half(scur[hf], m_use, pf[2 * hf], pf[2 * hf + 1]);
        l_run += ps;
#pragma unroll
        for (int ks = 0; ks < 2 * NH; ++ks) {
          vread(sa, ks, vv0);
          pv_mfma(vv0, pf[ks]);
        }
      }
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    using YES = std::integral_constant<bool, true>;
    using NO = std::integral_constant<bool, false>;
    int i = 0;
    for (; i + 4 < ntiles; i += 4) {  // steps i .. i+3 all have a next tile
      step(i, I0{}, I1{}, I3{}, YES{}, sa_buf, sb_buf);
      step(i + 1, I1{}, I2{}, I0{}, YES{}, sb_buf, sa_buf);
      step(i + 2, I2{}, I3{}, I1{}, YES{}, sa_buf, sb_buf);
      step(i + 3, I3{}, I0{}, I2{}, YES{}, sb_buf, sa_buf);
    }
    // 1..4 steps remain; the last has no next tile
    const int rem = ntiles - i;
    if (rem == 1) {
      step(i, I0{}, I1{}, I3{}, NO{}, sa_buf, sb_buf);
    } else if (rem == 2) {
      step(i, I0{}, I1{}, I3{}, YES{}, sa_buf, sb_buf);
      step(i + 1, I1{}, I2{}, I0{}, NO{}, sb_buf, sa_buf);
    } else if (rem == 3) {
      step(i, I0{}, I1{}, I3{}, YES{}, sa_buf, sb_buf);
      step(i + 1, I1{}, I2{}, I0{}, YES{}, sb_buf, sa_buf);
      step(i + 2, I2{}, I3{}, I1{}, NO{}, sa_buf, sb_buf);
    } else {
      step(i, I0{}, I1{}, I3{}, YES{}, sa_buf, sb_buf);
      step(i + 1, I1{}, I2{}, I0{}, YES{}, sb_buf, sa_buf);
      step(i + 2, I2{}, I3{}, I1{}, YES{}, sa_buf, sb_buf);
      step(i + 3, I3{}, I0{}, I2{}, NO{}, sb_buf, sa_buf);
    }

  }

  float l_tot = l_run + shfl_xor_f(l_run, 32);
  if (SPLIT) {
    // Merge the two key halves of each row group.  The ring is free once
    // every wave is past its last tile (the last wait was vmcnt 0).  O^T
    // group q of a lane (4 floats) goes to stage array q / (GPL/4).
    constexpr int QPA = R::GPL / 4;
    __syncthreads();
    if (kh0 == 1) {
#pragma unroll
      for (int q = 0; q < R::GPL; ++q) {
        const f32x4 v4 = {oacc[q / 4][4 * (q % 4)], oacc[q / 4][4 * (q % 4) + 1], oacc[q / 4][4 * (q % 4) + 2],
                          oacc[q / 4][4 * (q % 4) + 3]};
        *reinterpret_cast<f32x4*>(kst[q / QPA] + ((rg * QPA + q % QPA) * 64 + lane) * 16) = v4;
      }
      *reinterpret_cast<f32x2_t*>(v0 + (rg * 64 + lane) * 8) = f32x2_t{m_run, l_tot};
    }
    __syncthreads();
    if (kh0 == 1) return;
    const f32x2_t ml = *reinterpret_cast<const f32x2_t*>(v0 + (rg * 64 + lane) * 8);
    const float mn = __builtin_fmaxf(m_run, ml[0]);
    const float base = mn == -INFINITY ? 0.f : mn;
    const float a0 = __builtin_amdgcn_exp2f(m_run - base), a1 = __builtin_amdgcn_exp2f(ml[0] - base);
    l_tot = l_tot * a0 + ml[1] * a1;
    m_run = mn;
#pragma unroll
    for (int q = 0; q < R::GPL; ++q) {
      const f32x4 o1 = *reinterpret_cast<const f32x4*>(kst[q / QPA] + ((rg * QPA + q % QPA) * 64 + lane) * 16);
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[q / 4][4 * (q % 4) + e] = oacc[q / 4][4 * (q % 4) + e] * a0 + o1[e] * a1;
    }
  }
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
    // Split partial: the normalised output O/l (a convex combination of V
    // rows) in fp16, times 2^-e per row so that its largest magnitude lies
    // in [0.5, 1), plus the split's weight m + log2(l) (its row max and sum
    // in log2 units) and e, as two fp32 per row.  Fragment order: for each
    // (split, KV head, 32-row block) the lanes' O^T groups f = 4dt + q4 are
    // stored in pairs [f/2][lane] as 8 halves, so every store (and every
    // load of the combine) covers 1 KiB contiguously.
    float amax = 0.f;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int j = 0; j < 16; j += 2) amax = max3f(amax, __builtin_fabsf(oacc[dt][j]), __builtin_fabsf(oacc[dt][j + 1]));
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(amax), __float_as_uint(amax), false, false);
    amax = max3f(__uint_as_float(sw[0]), __uint_as_float(sw[1]), 0.f);
    const float inv_l = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const int ex = __builtin_amdgcn_frexp_expf(amax * inv_l);
    const float mul = __builtin_amdgcn_ldexpf(inv_l, -ex);
    const size_t blk = ((size_t)s * a.Hkv + g) * (a.Mpad / 32) + (row >> 5);
    u32x4* po = reinterpret_cast<u32x4*>(a.part_o) + blk * (R::GPL / 2) * 64 + lane;
#pragma unroll
    for (int k = 0; k < R::GPL / 2; ++k) {
      const int dt = k / 2, q0 = 8 * (k % 2);  // groups 2k, 2k+1: oacc[dt][q0 .. q0+8)
      u32x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = pack_f16x2(oacc[dt][q0 + 2 * e] * mul, oacc[dt][q0 + 2 * e + 1] * mul);
      po[k * 64] = h;
    }
    if (u == 0)
      *reinterpret_cast<f32x2_t*>(a.part_ml + (((size_t)s * a.Hkv + g) * a.Mpad + row) * 2) =
          f32x2_t{l_tot > 0.f ? m_run + __builtin_amdgcn_logf(l_tot) : -INFINITY, (float)ex};
  }
}

// Merge the splits of each query row:
// O = sum_s 2^(w_s - w) 2^e_s P_s / sum_s 2^(w_s - w) with w = max_s w_s,
// where w_s = m_s + log2(l_s) is the log2 weight of split s (its row max
// and sum), P_s the stored fp16 partial and 2^e_s its scale.  A split that
// saw no allowed key has w_s = -inf and gets weight zero.  One wave per
// (KV head, 32-row block, pair of O^T groups): lane (c, u) owns row c and
// the 8 columns 32(k/2) + 16(k%2) + 4u + {0..3, 8..11}.  Every load is
// issued before any arithmetic (one round trip to memory): splits past the
// count re-read the last split and get weight zero.
// Waves per combine workgroup: one, so that the partial reads spread over
// as many CUs as possible.  Main kernel plus combine per call, each pair
// timed in one process: at the Qwen3-8B shape (64 nodes, 4k prefix, 13
// splits) four waves 15.95 against two 15.75 us, two 15.28 against one
// 15.25 us; at the Qwen3-0.6B shape (32 nodes, 1k prefix, 9 splits) two
// 9.96 against one 9.74 us.
constexpr int kCombineWaves = 1;

template <int D, int SMAX>
__global__ __launch_bounds__(64 * kCombineWaves) void tree_attn_combine_kernel(AttnArgs a) {
  constexpr int NP = D / 16;  // group pairs per lane
  const int lane = threadIdx.x & 63;
  // Same XCD-aware order as the main kernel: the blocks that share
  // blockIdx % 8 take one contiguous range of (KV head, row block), the
  // range whose partials that XCD wrote, so the loads hit its L2.
  int b = blockIdx.x;
  if (gridDim.x % 8 == 0) b = (b % 8) * (gridDim.x / 8) + b / 8;
  const int wv = b * kCombineWaves + (threadIdx.x >> 6);
  const int nblk = a.Mpad / 32;
  if (wv >= a.Hkv * nblk * NP) return;
  const int k = wv % NP, blk = (wv / NP) % nblk, g = wv / (NP * nblk);
  const int c = lane & 31, u = lane >> 5;
  const int r = blk * 32 + c;
  if (r >= a.M) return;
  const size_t split_o = (size_t)a.Hkv * nblk * NP * 64;  // 16-byte units between consecutive splits
  const size_t split_ml = (size_t)a.Hkv * a.Mpad;         // rows between consecutive splits
  const u32x4* po = reinterpret_cast<const u32x4*>(a.part_o) + (((size_t)g * nblk + blk) * NP + k) * 64 + lane;
  const f32x2_t* pml = reinterpret_cast<const f32x2_t*>(a.part_ml) + (size_t)g * a.Mpad + r;
  f32x2_t ml[SMAX];
  u32x4 o[SMAX];
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {  // splits past the count re-read the last one (weight zero below)
    const int sc = min(s, a.splits - 1);
    ml[s] = pml[sc * split_ml];
    o[s] = po[sc * split_o];
  }
  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) m = s < a.splits ? __builtin_fmaxf(m, ml[s][0]) : m;
  const float base = m == -INFINITY ? 0.f : m;
  float den = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    const float wgt = s < a.splits ? __builtin_amdgcn_exp2f(ml[s][0] - base) : 0.f;
    den += wgt;
    const float wv2 = __builtin_amdgcn_ldexpf(wgt, (int)ml[s][1]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const f32x2_t h = unpack_f16x2(o[s][e]);
      acc[2 * e] += wv2 * h[0];
      acc[2 * e + 1] += wv2 * h[1];
    }
  }
  const float inv = 1.f / den;
  const int node = r / a.G, head = g * a.G + r % a.G;
  uint16_t* orow = a.out + ((size_t)node * a.Hq + head) * D + 32 * (k / 2) + 16 * (k % 2) + 4 * u;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    u32x2 pk;
    pk[0] = pack_bf16x2(acc[4 * h] * inv, acc[4 * h + 1] * inv);
    pk[1] = pack_bf16x2(acc[4 * h + 2] * inv, acc[4 * h + 3] * inv);
    *reinterpret_cast<u32x2*>(orow + 8 * h) = pk;
  }
}

// float32 path: one workgroup of 256 threads per (node, query head).  Keys
// go in chunks of 256, one key per thread: key j is cache row j (prefix
// rows, then node rows P + i, allowed when bit i of the node's ancestor mask
// is set).  Each thread scores its key against the query (in LDS), the
// block takes the chunk's max, and the probabilities go to LDS; then thread
// t accumulates column t % D of P V over the keys j = t / D (mod 256 / D),
// with the running max/sum of an online softmax across chunks.  The
// 256 / D column partials are added at the end.
template <int D>
__global__ __launch_bounds__(256) void tree_attn_f32_kernel(const float* q, const float* k, const float* v,
                                                            long long cap, int P, const int* P_dev, int N,
                                                            const uint64_t* mask, int W, int Hq, int Hkv,
                                                            float scale, float* out) {
  constexpr int NT = 256, PARTS = NT / D;
  __shared__ float qs[D];
  __shared__ float ps[NT];
  __shared__ float red[NT / 64];
  __shared__ float opart[NT];
  if (P_dev) P = min(max(*P_dev, 0), P);
  const int node = blockIdx.x / Hq, head = blockIdx.x % Hq;
  const int g = head / (Hq / Hkv);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float sl2 = scale * 1.4426950408889634f;
  if (t < D) qs[t] = q[((size_t)node * Hq + head) * D + t] * sl2;
  const float* kb = k + (size_t)g * cap * D;
  const float* vb = v + (size_t)g * cap * D;
  const uint64_t* mrow = mask + (size_t)node * W;
  const int col = t % D, part = t / D;
  float m_run = -INFINITY, l_run = 0.f, o = 0.f;
  __syncthreads();
  for (int c0 = 0; c0 < P + N; c0 += NT) {
    const int j = c0 + t;
    bool ok = j < P;
    if (!ok && j < P + N) ok = (mrow[(j - P) >> 6] >> ((j - P) & 63)) & 1ull;
    float sc = -INFINITY;
    if (ok) {
      const float4* kr = reinterpret_cast<const float4*>(kb + (size_t)j * D);
      float a0 = 0.f, a1 = 0.f;
#pragma unroll
      for (int d4 = 0; d4 < D / 4; d4 += 2) {
        const float4 x = kr[d4], y = kr[d4 + 1];
        a0 += x.x * qs[4 * d4] + x.y * qs[4 * d4 + 1] + x.z * qs[4 * d4 + 2] + x.w * qs[4 * d4 + 3];
        a1 += y.x * qs[4 * d4 + 4] + y.y * qs[4 * d4 + 5] + y.z * qs[4 * d4 + 6] + y.w * qs[4 * d4 + 7];
      }
      sc = a0 + a1;
    }
    float mx = sc;
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, shfl_xor_f(mx, off));
    if (lane == 0) red[wave] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const float m_new = fmaxf(m_run, mx);  // finite: every node sees itself
    const float alpha = exp2f(m_run - m_new);
    const float p = ok ? exp2f(sc - m_new) : 0.f;
    ps[t] = p;
    float sum = p;
    for (int off = 32; off > 0; off >>= 1) sum += shfl_xor_f(sum, off);
    __syncthreads();  // ps complete; every wave has read red
    if (lane == 0) red[wave] = sum;
    __syncthreads();
    l_run = l_run * alpha + ((red[0] + red[1]) + (red[2] + red[3]));
    m_run = m_new;
    float acc = 0.f;
    const int nk = min(NT, P + N - c0);
    for (int jj = part; jj < nk; jj += PARTS) {
      const float pj = ps[jj];
      if (pj != 0.f) acc += pj * vb[(size_t)(c0 + jj) * D + col];  // rows of keys not allowed are not read
    }
    o = o * alpha + acc;
    __syncthreads();  // before the next chunk overwrites ps and red
  }
  opart[t] = o;
  __syncthreads();
  if (t < D) {
    float s = 0.f;
#pragma unroll
    for (int pp = 0; pp < PARTS; ++pp) s += opart[pp * D + t];
    out[((size_t)node * Hq + head) * D + t] = s / l_run;
  }
}

// The combine kernel loads exactly the splits there are (up to 16; more in
// groups of 4): each padding slot is one more load per lane, and the merge
// is bound by its loads.
template <int D, int S>
void launch_combine_n(dim3 grid, hipStream_t st, const AttnArgs& a) {
  tree_attn_combine_kernel<D, S><<<grid, 64 * kCombineWaves, 0, st>>>(a);
}
template <int D>
void launch_combine(int splits, dim3 grid, hipStream_t st, const AttnArgs& a) {
  switch (splits) {
    case 2: return launch_combine_n<D, 2>(grid, st, a);
    case 3: return launch_combine_n<D, 3>(grid, st, a);
    case 4: return launch_combine_n<D, 4>(grid, st, a);
    case 5: return launch_combine_n<D, 5>(grid, st, a);
    case 6: return launch_combine_n<D, 6>(grid, st, a);
    case 7: return launch_combine_n<D, 7>(grid, st, a);
    case 8: return launch_combine_n<D, 8>(grid, st, a);
    case 9: return launch_combine_n<D, 9>(grid, st, a);
    case 10: return launch_combine_n<D, 10>(grid, st, a);
    case 11: return launch_combine_n<D, 11>(grid, st, a);
    case 12: return launch_combine_n<D, 12>(grid, st, a);
    case 13: return launch_combine_n<D, 13>(grid, st, a);
    case 14: return launch_combine_n<D, 14>(grid, st, a);
    case 15: return launch_combine_n<D, 15>(grid, st, a);
    case 16: return launch_combine_n<D, 16>(grid, st, a);
    default:
      if (splits <= 20) return launch_combine_n<D, 20>(grid, st, a);
      if (splits <= 24) return launch_combine_n<D, 24>(grid, st, a);
      if (splits <= 28) return launch_combine_n<D, 28>(grid, st, a);
      return launch_combine_n<D, 32>(grid, st, a);
  }
}

struct Plan {
  int waves, row_blocks, Mpad, tiles_prefix, tiles_total, splits, tps;
  size_t ws_bytes;
};

// force_splits > 0 replaces the planner's split count (tests and tuning).
Plan make_plan(int N, int Hq, int Hkv, int D, int P, ooo_dtype dt, int force_splits) {
  Plan p{};
  if (dt != OOO_BF16) return p;
  const int G = Hq / Hkv;
  const int M = N * G;
  p.waves = M <= 64 ? 2 : 4;  // waves of 32 query rows
  const int BM = 32 * p.waves;
  p.row_blocks = (M + BM - 1) / BM;
  p.Mpad = p.row_blocks * BM;
  p.tiles_prefix = (P + kTile - 1) / kTile;
  p.tiles_total = p.tiles_prefix + (N + kTile - 1) / kTile;
  // Split count: as many workgroups as fit on the CUs at once, balancing the
  // tiles of the busiest split against the partials every split adds (an
  // empirical cost of about 1.3 us per 64-key tile and 0.5 us per split of
  // 128-row blocks, half that for 64-row blocks, whose partials are half
  // the size: at 32 nodes, 2 query heads per KV head and a 1k prefix, 9
  // splits take 9.96 us per call and the 6 of the 128-row cost 10.8 us).
  // Units of 0.05 us.
  const int base = Hkv * p.row_blocks;
  const int max_splits = device_cus() / base > 1 ? device_cus() / base : 1;
  const int split_cost = p.waves == 2 ? 5 : 10;
  int splits = 1, best = INT32_MAX;
  for (int sc = 1; sc <= max_splits && sc <= p.tiles_total; ++sc) {
    const int cost = 26 * ((p.tiles_total + sc - 1) / sc) + split_cost * sc;
    if (cost < best) best = cost, splits = sc;
  }
  if (force_splits > 0) splits = force_splits;
  if (splits > 32) splits = 32;
  if (splits > p.tiles_total) splits = p.tiles_total;
  if (splits < 1) splits = 1;
  // fixed-size runs of tiles; the last run may be shorter
  p.tps = (p.tiles_total + splits - 1) / splits;
  p.splits = (p.tiles_total + p.tps - 1) / p.tps;
  if (p.splits > 1)
    p.ws_bytes = (size_t)p.splits * Hkv * p.Mpad * (size_t)D * 2 + (size_t)p.splits * Hkv * p.Mpad * 8 + 256;
  return p;
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" size_t ooo_tree_attn_workspace_ex(int32_t n_nodes, int32_t n_q_heads, int32_t n_kv_heads,
                                             int32_t head_dim, int32_t prefix_len, ooo_dtype dt,
                                             int32_t force_splits) {
  if (n_nodes < 1 || n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads || prefix_len < 0) return 0;
  return make_plan(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt, force_splits).ws_bytes;
}

extern "C" size_t ooo_tree_attn_workspace(int32_t n_nodes, int32_t n_q_heads, int32_t n_kv_heads,
                                          int32_t head_dim, int32_t prefix_len, ooo_dtype dt) {
  return ooo_tree_attn_workspace_ex(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt, 0);
}

extern "C" int ooo_tree_attn_ex(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                                int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                                const uint64_t* anc_mask, int32_t mask_words, int32_t n_q_heads,
                                int32_t n_kv_heads, int32_t head_dim, float scale, ooo_dtype dt, void* out,
                                void* workspace, size_t ws_bytes, void* stream, int32_t force_splits,
                                int32_t variant) {
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
  OOO_REQUIRE(force_splits >= 0 && (variant == 0 || variant == 1), OOO_ERR_INVALID,
              "ooo_tree_attn: force_splits (%d) must be >= 0 and variant (%d) 0 or 1", force_splits, variant);
  OOO_REQUIRE(head_dim == 64 || head_dim == 128, OOO_ERR_UNSUPPORTED,
              "ooo_tree_attn: head_dim %d not supported (64 or 128)", head_dim);
  OOO_REQUIRE((int64_t)n_nodes * n_q_heads * head_dim * 2 < (1LL << 32), OOO_ERR_UNSUPPORTED,
              "ooo_tree_attn: Q of %d nodes x %d heads exceeds 4 GiB", n_nodes, n_q_heads);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int G = n_q_heads / n_kv_heads;

  if (dt == OOO_F32) {
    const dim3 grid(n_nodes * n_q_heads);
    if (head_dim == 64)
      tree_attn_f32_kernel<64><<<grid, 256, 0, st>>>((const float*)q, (const float*)k_cache, (const float*)v_cache,
                                                    cap, prefix_len, prefix_len_dev, n_nodes, anc_mask, mask_words,
                                                    n_q_heads, n_kv_heads, scale, (float*)out);
    else
      tree_attn_f32_kernel<128><<<grid, 256, 0, st>>>((const float*)q, (const float*)k_cache, (const float*)v_cache,
                                                     cap, prefix_len, prefix_len_dev, n_nodes, anc_mask,
                                                     mask_words, n_q_heads, n_kv_heads, scale, (float*)out);
  } else {
    const Plan p = make_plan(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt, force_splits);
    OOO_REQUIRE(ws_bytes >= p.ws_bytes && (p.ws_bytes == 0 || workspace), OOO_ERR_CAPACITY,
                "ooo_tree_attn: workspace of %zu bytes needed (got %zu)", p.ws_bytes, ws_bytes);
    AttnArgs a{};
    a.q = (const uint16_t*)q;
    a.k = (const uint16_t*)k_cache;
    a.v = (const uint16_t*)v_cache;
    a.cap = cap;
    a.P = prefix_len;
    a.P_dev = prefix_len_dev;
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
    a.tps = p.tps;
    if (p.splits > 1) {
      a.part_o = (uint32_t*)workspace;
      a.part_ml = (float*)((uint8_t*)workspace + (size_t)p.splits * n_kv_heads * p.Mpad * head_dim * 2);
    }
    const dim3 grid(n_kv_heads * p.row_blocks * p.splits);
    // head_dim 128 runs the key-split kernel (two waves per row group);
    // variant 1 selects the one-wave pipelined kernel instead.
    if (head_dim == 128 && variant == 0) {
      if (p.waves == 2) tree_attn_bf16_kernel<128, 2, true><<<grid, 256, 0, st>>>(a);
      else tree_attn_bf16_kernel<128, 4, true><<<grid, 512, 0, st>>>(a);
    } else if (head_dim == 128) {
      if (p.waves == 2) tree_attn_bf16_kernel<128, 2, false><<<grid, 128, 0, st>>>(a);
      else tree_attn_bf16_kernel<128, 4, false><<<grid, 256, 0, st>>>(a);
    } else {
      if (p.waves == 2) tree_attn_bf16_kernel<64, 2, false><<<grid, 128, 0, st>>>(a);
      else tree_attn_bf16_kernel<64, 4, false><<<grid, 256, 0, st>>>(a);
    }
    if (p.splits > 1) {
      const int waves = n_kv_heads * (p.Mpad / 32) * (head_dim / 16);
      const dim3 cgrid((waves + kCombineWaves - 1) / kCombineWaves);
      if (head_dim == 128) launch_combine<128>(p.splits, cgrid, st, a);
      else launch_combine<64>(p.splits, cgrid, st, a);
    }
  }
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_tree_attn: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

// Scratch of ooo_tree_attn_noalloc: one copy per GPU, held until the
// process ends.  Host code never passes `scratch` itself to a kernel (in
// host code it is a stand-in, not a device address): the device address is
// looked up once per device with hipGetSymbolAddress.
constexpr size_t kNoAllocScratchBytes = 16u << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
}  // namespace

extern "C" size_t ooo_tree_attn_noalloc_scratch_bytes(void) { return kNoAllocScratchBytes; }

extern "C" int ooo_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                                     int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                                     const uint64_t* anc_mask, int32_t mask_words, int32_t n_q_heads,
                                     int32_t n_kv_heads, int32_t head_dim, float scale, ooo_dtype dt, void* out,
                                     void* stream) {
  const size_t need =
      (n_nodes >= 1 && n_kv_heads >= 1 && n_q_heads >= 1 && n_q_heads % n_kv_heads == 0 && prefix_len >= 0)
          ? make_plan(n_nodes, n_q_heads, n_kv_heads, head_dim, prefix_len, dt, 0).ws_bytes
          : 0;
  OOO_REQUIRE(need <= kNoAllocScratchBytes, OOO_ERR_CAPACITY,
              "ooo_tree_attn_noalloc: this shape needs %zu bytes of scratch; the built-in scratch holds %zu",
              need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if (need > 0) {
    int dev = -1;
    const hipError_t ge = hipGetDevice(&dev);
    OOO_REQUIRE(ge == hipSuccess && dev >= 0 && dev < kMaxDevices, OOO_ERR_HIP,
                "ooo_tree_attn_noalloc: no current device (%s)", hipGetErrorString(ge));
    std::call_once(g_scratch_once[dev], [dev] {
      g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
    });
    OOO_REQUIRE(g_scratch_err[dev] == hipSuccess && g_scratch_ptr[dev], OOO_ERR_HIP,
                "ooo_tree_attn_noalloc: scratch address on device %d: %s", dev,
                hipGetErrorString(g_scratch_err[dev]));
    ws = g_scratch_ptr[dev];
  }
  return ooo_tree_attn_ex(q, k_cache, v_cache, cap, prefix_len, prefix_len_dev, n_nodes, anc_mask, mask_words,
                          n_q_heads, n_kv_heads, head_dim, scale, dt, out, ws, need > 0 ? kNoAllocScratchBytes : 0,
                          stream, 0, 0);
}

extern "C" int ooo_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t cap,
                             int32_t prefix_len, const int32_t* prefix_len_dev, int32_t n_nodes,
                             const uint64_t* anc_mask, int32_t mask_words, int32_t n_q_heads, int32_t n_kv_heads,
                             int32_t head_dim, float scale, ooo_dtype dt, void* out, void* workspace,
                             size_t ws_bytes, void* stream) {
  return ooo_tree_attn_ex(q, k_cache, v_cache, cap, prefix_len, prefix_len_dev, n_nodes, anc_mask, mask_words,
                          n_q_heads, n_kv_heads, head_dim, scale, dt, out, workspace, ws_bytes, stream, 0, 0);
}
