// Weight-streaming core shared by the LM head (lmhead.hip) and the decoder
// projections (linear.hip): products W X^T of a weight W that is streamed
// once from HBM with a few node rows X (N <= 256) that every block re-reads
// from L2.
//  * W is cut into 128-row tiles and 64-column chunks; a chunk is 16 KiB,
//    four 32-row slots of 4 KiB.  In the packed layout (ooo_lmhead_pack)
//    chunk (t, kc) is one contiguous 16 KiB block, already swizzled; in the
//    row layout (nn.Linear) a slot is gathered row by row.
//  * In LDS the 16-byte piece p of row r sits at piece p ^ ((r / 2) % 8).
//    A 128-byte row covers half of gfx950's 64 LDS banks, so even and odd
//    rows fall in opposite halves, and a 16-byte read serves 16 lanes (16
//    rows, one piece) at a time: with the XOR by (r / 2) % 8 the eight rows
//    in each half read eight different pieces, all 64 banks once.  (An XOR
//    by r % 8 gave rows r and r + 8 the same banks: a 2-way conflict on
//    every fragment read.)
//  * Seven waves per block: four compute waves own 32 W rows each; two
//    loader waves DMA the W slots (two each) and a third the X chunk into a
//    ring of NS stages, NS - 1 chunks requested ahead of the one consumed.
//    Wider node tiles need more X bytes per stage, so fewer stages fit.
//  * The contraction index inside a chunk follows the pieces: MFMA k-step s,
//    lane half u, element e is k = 8 (2s + u) + e for both operands.
#pragma once

#include "device_common.h"

namespace ooo {

constexpr int kStreamRows = 128;  // W rows per tile (4 compute waves x 32)
constexpr int kStreamThreads = 448;  // 4 compute waves + 2 W loaders + 1 X loader

// physical piece of logical piece p in LDS row r (and in the packed layout)
__device__ __forceinline__ int piece_swz(int r) { return (r >> 1) & 7; }

template <int NB>
struct StreamRing {
  static constexpr int XR = 32 * NB;              // node rows staged (padded)
  static constexpr int WS = kStreamRows * 128;    // bytes of a W chunk
  static constexpr int XS = XR * 128;             // bytes of an X chunk
  static constexpr int NS = NB == 1 ? 7 : NB == 2 ? 6 : NB == 4 ? 4 : 3;
  static constexpr int XREG = NS * WS;            // start of the X stages
  static constexpr int BYTES = NS * (WS + XS);
  static constexpr int WDMA = WS / 1024 / 2;      // DMA instructions per W chunk and W loader
  static constexpr int XDMA = XS / 1024;          // ... per X chunk
  static_assert((NS - 2) * WDMA <= 63 && (NS - 2) * XDMA <= 63, "vmcnt range");
  static_assert(BYTES <= 160 * 1024, "LDS capacity");
};

// wait until at most `ahead` chunks of PER DMA instructions are pending
template <int PER, int MAXA>
__device__ __forceinline__ void wait_chunks(int ahead) {
  static_assert(MAXA <= 5, "ring depth");
  if (MAXA >= 5 && ahead >= 5) wait_vmcnt<(MAXA >= 5 ? 5 * PER : 0)>();
  else if (MAXA >= 4 && ahead == 4) wait_vmcnt<(MAXA >= 4 ? 4 * PER : 0)>();
  else if (MAXA >= 3 && ahead == 3) wait_vmcnt<(MAXA >= 3 ? 3 * PER : 0)>();
  else if (MAXA >= 2 && ahead == 2) wait_vmcnt<(MAXA >= 2 ? 2 * PER : 0)>();
  else if (ahead == 1) wait_vmcnt<PER>();
  else wait_vmcnt<0>();
}

// One 32-row W slot (4 KiB at dst).  Packed: src is the slot's 4 KiB run
// plus lane * 8 elements (a slot whose group is empty passes an L2-resident
// address with step 0, so every chunk has the same instruction count).
__device__ __forceinline__ void dma_w_slot_packed(const uint16_t* src, int step, uint8_t* dst) {
#pragma unroll
  for (int jj = 0; jj < 4; ++jj)
    __builtin_amdgcn_global_load_lds(OOO_GLB(src + (step ? jj * 512 : 0)), OOO_LDS(dst + jj * 1024), 16, 0,
                                     kStreamOnce);
}
// Row layout: rows row0 .. row0 + 31 of W[rows][ld] (clamped to the last
// row), columns 64 kc .. 64 kc + 63; lane = (row within an instruction,
// physical piece).
__device__ __forceinline__ void dma_w_slot_rows(const uint16_t* W, long long ld, int row0, int rows, int kc,
                                                uint8_t* dst, int lane) {
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const int r = 8 * jj + lane / 8;
    const int pc = (lane % 8) ^ piece_swz(r);
    const int row = min(row0 + r, rows - 1);
    __builtin_amdgcn_global_load_lds(OOO_GLB(W + (size_t)row * ld + kc * 64 + pc * 8), OOO_LDS(dst + jj * 1024),
                                     16, 0, kStreamOnce);
  }
}

// X chunk kc of X[N][ld] (rows padded to 32 NB by repeating the last row).
template <int NB>
__device__ __forceinline__ void dma_x_chunk(const uint16_t* X, int N, long long ld, int kc, uint8_t* dst, int lane) {
#pragma unroll
  for (int j = 0; j < StreamRing<NB>::XDMA; ++j) {
    const int r = 8 * j + lane / 8;
    const int pc = (lane % 8) ^ piece_swz(r);
    const int row = min(r, N - 1);
    __builtin_amdgcn_global_load_lds(OOO_GLB(X + (size_t)row * ld + kc * 64 + pc * 8), OOO_LDS(dst + j * 1024), 16, 0,
                                     0);
  }
}

// A loader wave's stream of `total` chunks: chunks 0 .. NS - 2 up front,
// then for every chunk q: wait for this wave's share of chunk q, the block
// barrier (every share landed, and the compute waves are done with chunk
// q - 1), then request chunk q + NS - 1 into the stage chunk q - 1 used.
// issue(q, stage) issues this wave's PER DMA instructions of chunk q.
template <int NS, int PER, class Issue>
__device__ __forceinline__ void loader_stream(int total, Issue&& issue) {
  for (int q = 0; q < NS - 1 && q < total; ++q) issue(q, q);
  for (int q = 0; q < total; ++q) {
    wait_chunks<PER, NS - 2>(min(NS - 2, total - 1 - q));
    wg_barrier();
    if (q + NS - 1 < total) issue(q + NS - 1, (q + NS - 1) % NS);
  }
}

// LDS byte offsets of compute lane (c, u)'s fragments in a W or X stage:
// piece 2s + u of row c (swizzled), for the k-steps s of a chunk.
__device__ __forceinline__ void frag_offsets(int lane, uint32_t (&off)[4]) {
  const int c = lane & 31, u = lane >> 5;
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) off[s4] = c * 128 + (((2 * s4 + u) ^ piece_swz(c)) << 4);
}

// One chunk of a compute wave: acc[nb] += (its 32 W rows at Ws) x (node
// rows 32 nb .. 32 nb + 31 at Xs)^T.  acc[nb][j] then belongs to W row
// 8 (j / 4) + 4 u + j % 4 of the wave's 32 and node 32 nb + c.
template <int NB>
__device__ __forceinline__ void chunk_mfma(const uint8_t* Ws, const uint8_t* Xs, const uint32_t (&off)[4],
                                           f32x16 (&acc)[NB]) {
  bf16x8 af[4], bf[NB][4];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    af[s4] = as_bf16x8(*reinterpret_cast<const u32x4*>(Ws + off[s4]));
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bf[nb][s4] = as_bf16x8(*reinterpret_cast<const u32x4*>(Xs + nb * 4096 + off[s4]));
  }
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = mfma32(af[s4], bf[nb][s4], acc[nb]);
}

}  // namespace ooo
