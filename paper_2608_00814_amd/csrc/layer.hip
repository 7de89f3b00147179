// Decoder layer around the verification path.  The paper scores the whole
// candidate tree with one forward pass of the target (Section 4.5) and runs
// Qwen3 targets (Section 5); the layer is the standard Qwen3 decoder layer.
// The tree-specific part is the rotary position: node i sits at P +
// depth[i], the position sequential decoding of its own root path gives it,
// and its key/value row goes to cache row P + i (the tree attention reads it
// there; compaction later moves the accepted rows).
//
//  * ooo_embed_rows     residual rows h[N][H] (fp32) = embedding[token]
//  * ooo_rmsnorm        x = h / sqrt(mean(h^2) + eps) * w, fp32 in, bf16 out
//  * ooo_qk_norm_rope   per-head RMSNorm of q and k, rotation at P + depth,
//                       q to a [N][Hq][D] buffer, k and v to the cache rows
//  * ooo_swiglu         silu(gate) * up
// The projections between them are ooo_linear (linear.hip).
#include <math.h>

#include "device_common.h"
#include "ooo_internal.h"
#include "rope.h"

namespace ooo {
namespace {

// ---------------------------------------------------------------- embedding
// One block per node, 16-byte loads (8 bf16); a token outside [0, V)
// yields NaN rows (visible, not silently clamped).  H % 8 == 0.
__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* __restrict__ table,
                                                    const int32_t* __restrict__ tokens, int H, int V,
                                                    float* __restrict__ h) {
  const int n = blockIdx.x;
  const int t = tokens[n];
  const bool ok = t >= 0 && t < V;
  for (int c = threadIdx.x * 8; c < H; c += 256 * 8) {
    f32x4 lo = {__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf("")}, hi = lo;
    if (ok) {
      const u32x4 v = ld16(table + (size_t)t * H + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const f32x2_t f = {__uint_as_float(v[e] << 16), __uint_as_float(v[e] & 0xFFFF0000u)};
        if (e < 2) {
          lo[2 * e] = f[0];
          lo[2 * e + 1] = f[1];
        } else {
          hi[2 * e - 4] = f[0];
          hi[2 * e - 3] = f[1];
        }
      }
    }
    *reinterpret_cast<f32x4*>(h + (size_t)n * H + c) = lo;
    *reinterpret_cast<f32x4*>(h + (size_t)n * H + c + 4) = hi;
  }
}

// ------------------------------------------------------------------ RMSNorm
// One block (256 threads) per row; the row (dim <= 8192, dim % 4 == 0) is
// read once with all 16-byte loads issued up front and kept in registers:
// sum of squares in fp32, then out = h * (1 / sqrt(ss / H + eps)) * w
// rounded to bf16.
constexpr int kNormVec = 8;  // float4 per thread
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h, const uint16_t* __restrict__ w,
                                                      int H, float eps, uint16_t* __restrict__ out) {
  __shared__ float part[4];
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* row = h + (size_t)n * H;
  f32x4 v[kNormVec];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kNormVec; ++i) {
    const int c = 4 * (threadIdx.x + 256 * i);
    v[i] = c < H ? *reinterpret_cast<const f32x4*>(row + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int i = 0; i < kNormVec; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) ss = __builtin_fmaf(v[i][e], v[i][e], ss);
  for (int off = 32; off > 0; off >>= 1) ss += shfl_xor_f(ss, off);
  if (lane == 0) part[wave] = ss;
  __syncthreads();
  const float tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float r = 1.f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int i = 0; i < kNormVec; ++i) {
    const int c = 4 * (threadIdx.x + 256 * i);
    if (c < H) {
      const u32x2 wv = *reinterpret_cast<const u32x2*>(w + c);
      u32x2 o;
      o[0] = pack_bf16x2(v[i][0] * r * __uint_as_float(wv[0] << 16), v[i][1] * r * __uint_as_float(wv[0] & 0xFFFF0000u));
      o[1] = pack_bf16x2(v[i][2] * r * __uint_as_float(wv[1] << 16), v[i][3] * r * __uint_as_float(wv[1] & 0xFFFF0000u));
      *reinterpret_cast<u32x2*>(out + (size_t)n * H + c) = o;
    }
  }
}

// ------------------------------------------------------ QK norm and rotation
// Block (node n, 16 heads), one wave per head: every load of the block is
// issued at once.  Lane j < D/2 owns the rotate-half pair (j, j + D/2); its
// rotation angle (P + depth[n]) * theta^(-2j/D) is formed in double
// precision and reduced by multiples of 2 pi before a float sine/cosine.  Heads [0, Hq) are queries, [Hq, Hq + Hkv) keys,
// [Hq + Hkv, Hq + 2 Hkv) values (copied to the cache unchanged).  A null norm
// weight skips that norm (models without QK norms).
template <int D>
__global__ __launch_bounds__(1024) void qk_norm_rope_kernel(const uint16_t* __restrict__ qkv,
                                                           const uint16_t* __restrict__ q_norm,
                                                           const uint16_t* __restrict__ k_norm, float eps,
                                                           const int32_t* __restrict__ depth, int P,
                                                           const int32_t* __restrict__ P_dev, RopeFreq fr,
                                                           int Hq, int Hkv, uint16_t* __restrict__ q_out,
                                                           uint16_t* __restrict__ k_cache,
                                                           uint16_t* __restrict__ v_cache, long long cap) {
  constexpr int HALF = D / 2;
  if (P_dev) P = min(max(*P_dev, 0), P);  // device prefix, bounded by the launch value
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nh = Hq + 2 * Hkv;
  const int hh = blockIdx.y * 16 + wave;  // this wave's head
  if (hh >= nh) return;
  const uint16_t* src = qkv + (size_t)n * nh * D;
  const long long row = (long long)P + n;  // node n's cache row
  const bool act = lane < HALF;
  float cs = 1.f, sn = 0.f;
  if (act) rope_sincos(P + depth[n], fr.f[lane], sn, cs);
  {
    const uint16_t* hr = src + (size_t)hh * D;
    if (hh >= Hq + Hkv) {
      const int g = hh - Hq - Hkv;
      uint16_t* dst = v_cache + ((size_t)g * cap + row) * D;
      if (act) {
        dst[lane] = hr[lane];
        dst[lane + HALF] = hr[lane + HALF];
      }
      return;
    }
    const bool is_q = hh < Hq;
    float a = act ? bf16_bits_to_f32(hr[lane]) : 0.f;
    float b = act ? bf16_bits_to_f32(hr[lane + HALF]) : 0.f;
    norm_rotate(a, b, act, is_q ? q_norm : k_norm, eps, D, lane, cs, sn);
    uint16_t* dst = is_q ? q_out + ((size_t)n * Hq + hh) * D : k_cache + ((size_t)(hh - Hq) * cap + row) * D;
    if (act) {
      dst[lane] = f32_to_bf16_bits(a);
      dst[lane + HALF] = f32_to_bf16_bits(b);
    }
  }
}

// ------------------------------------------------------------------- SwiGLU
// out[n][j] = silu(gu[n][j]) * gu[n][I + j]: the gate rows come first in the
// fused projection, then the up rows.
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ gu, int N, int I,
                                                     uint16_t* __restrict__ out) {
  const long long total = (long long)N * I;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
    const long long n = e / I, j = e - n * I;
    const float g = gu[n * 2 * I + j], u = gu[n * 2 * I + I + j];
    out[e] = f32_to_bf16_bits(g / (1.f + expf(-g)) * u);
  }
}

}  // namespace
}  // namespace ooo

using namespace ooo;

extern "C" int ooo_embed_rows(const void* table, const int32_t* tokens, int32_t n_nodes, int32_t hidden_dim,
                              int32_t vocab, float* h, void* stream) {
  OOO_REQUIRE(table && tokens && h, OOO_ERR_INVALID, "ooo_embed_rows: null pointer");
  OOO_REQUIRE(n_nodes >= 1 && hidden_dim >= 1 && vocab >= 1, OOO_ERR_INVALID, "ooo_embed_rows: sizes must be positive");
  OOO_REQUIRE(hidden_dim % 8 == 0, OOO_ERR_UNSUPPORTED, "ooo_embed_rows: hidden_dim %% 8 != 0");
  embed_kernel<<<n_nodes, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>((const uint16_t*)table, tokens, hidden_dim,
                                                                          vocab, h);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_embed_rows: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_rmsnorm(const float* h, const void* weight, int32_t n_rows, int32_t dim, float eps, void* out,
                           void* stream) {
  OOO_REQUIRE(h && weight && out, OOO_ERR_INVALID, "ooo_rmsnorm: null pointer");
  OOO_REQUIRE(n_rows >= 1 && dim >= 1, OOO_ERR_INVALID, "ooo_rmsnorm: sizes must be positive");
  OOO_REQUIRE(eps >= 0.f, OOO_ERR_INVALID, "ooo_rmsnorm: eps must be >= 0");
  OOO_REQUIRE(dim % 4 == 0 && dim <= 4 * 256 * kNormVec, OOO_ERR_UNSUPPORTED,
              "ooo_rmsnorm: dim %d not supported (a multiple of 4, at most %d)", dim, 4 * 256 * kNormVec);
  rmsnorm_kernel<<<n_rows, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(h, (const uint16_t*)weight, dim, eps,
                                                                           (uint16_t*)out);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_rmsnorm: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_qk_norm_rope(const void* qkv, const void* q_norm, const void* k_norm, float eps,
                                const int32_t* depth, int32_t n_nodes, int32_t prefix_len,
                                const int32_t* prefix_len_dev, double rope_theta,
                                int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, void* q_out,
                                void* k_cache, void* v_cache, int64_t cap, void* stream) {
  OOO_REQUIRE(qkv && depth && q_out && k_cache && v_cache, OOO_ERR_INVALID, "ooo_qk_norm_rope: null pointer");
  OOO_REQUIRE(n_nodes >= 1 && prefix_len >= 0 && n_q_heads >= 1 && n_kv_heads >= 1, OOO_ERR_INVALID,
              "ooo_qk_norm_rope: sizes must be positive");
  OOO_REQUIRE((int64_t)prefix_len + n_nodes <= cap, OOO_ERR_INVALID,
              "ooo_qk_norm_rope: prefix_len + n_nodes (%lld) exceeds cap (%lld)", (long long)prefix_len + n_nodes,
              (long long)cap);
  OOO_REQUIRE(rope_theta > 0.0 && eps >= 0.f, OOO_ERR_INVALID, "ooo_qk_norm_rope: rope_theta must be > 0");
  OOO_REQUIRE(head_dim == 64 || head_dim == 128, OOO_ERR_UNSUPPORTED,
              "ooo_qk_norm_rope: head_dim %d not supported (64 or 128)", head_dim);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const RopeFreq fr = rope_freq(rope_theta, head_dim);
  const dim3 grid(n_nodes, (n_q_heads + 2 * n_kv_heads + 15) / 16);
  if (head_dim == 128)
    qk_norm_rope_kernel<128><<<grid, 1024, 0, st>>>((const uint16_t*)qkv, (const uint16_t*)q_norm,
                                                      (const uint16_t*)k_norm, eps, depth, prefix_len, prefix_len_dev, fr,
                                                      n_q_heads, n_kv_heads, (uint16_t*)q_out, (uint16_t*)k_cache,
                                                      (uint16_t*)v_cache, cap);
  else
    qk_norm_rope_kernel<64><<<grid, 1024, 0, st>>>((const uint16_t*)qkv, (const uint16_t*)q_norm,
                                                     (const uint16_t*)k_norm, eps, depth, prefix_len, prefix_len_dev, fr,
                                                     n_q_heads, n_kv_heads, (uint16_t*)q_out, (uint16_t*)k_cache,
                                                     (uint16_t*)v_cache, cap);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_qk_norm_rope: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_swiglu(const float* gate_up, int32_t n_rows, int32_t intermediate, void* out, void* stream) {
  OOO_REQUIRE(gate_up && out, OOO_ERR_INVALID, "ooo_swiglu: null pointer");
  OOO_REQUIRE(n_rows >= 1 && intermediate >= 1, OOO_ERR_INVALID, "ooo_swiglu: sizes must be positive");
  const long long total = (long long)n_rows * intermediate;
  const int blocks = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
  swiglu_kernel<<<blocks, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(gate_up, n_rows, intermediate,
                                                                          (uint16_t*)out);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_swiglu: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}
