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

namespace ooo {
namespace {

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float v) {
  return (uint16_t)(pack_bf16x2(v, 0.f) & 0xFFFFu);
}

// ---------------------------------------------------------------- embedding
// One block per node; a token outside [0, V) yields NaN rows (visible, not
// silently clamped).
__global__ __launch_bounds__(256) void embed_kernel(const uint16_t* __restrict__ table,
                                                    const int32_t* __restrict__ tokens, int H, int V,
                                                    float* __restrict__ h) {
  const int n = blockIdx.x;
  const int t = tokens[n];
  const bool ok = t >= 0 && t < V;
  for (int c = threadIdx.x; c < H; c += blockDim.x)
    h[(size_t)n * H + c] = ok ? bf16_bits_to_f32(table[(size_t)t * H + c]) : __builtin_nanf("");
}

// ------------------------------------------------------------------ RMSNorm
// One block (256 threads) per row: sum of squares in fp32, then
// out = h * (1 / sqrt(ss / H + eps)) * w rounded to bf16.
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h, const uint16_t* __restrict__ w,
                                                      int H, float eps, uint16_t* __restrict__ out) {
  __shared__ float part[4];
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* row = h + (size_t)n * H;
  float ss = 0.f;
  for (int c = threadIdx.x; c < H; c += 256) {
    const float v = row[c];
    ss = __builtin_fmaf(v, v, ss);
  }
  for (int off = 32; off > 0; off >>= 1) ss += shfl_xor_f(ss, off);
  if (lane == 0) part[wave] = ss;
  __syncthreads();
  const float tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float r = 1.f / sqrtf(tot / (float)H + eps);
  for (int c = threadIdx.x; c < H; c += 256)
    out[(size_t)n * H + c] = f32_to_bf16_bits(row[c] * r * bf16_bits_to_f32(w[c]));
}

// ------------------------------------------------------ QK norm and rotation
// One block per node, one wave per head at a time.  Lane j < D/2 owns the
// rotate-half pair (j, j + D/2) of every head, so its rotation angle
// (P + depth[n]) * theta^(-2j/D) is computed once, in double precision, and
// reused for all heads.  Heads [0, Hq) are queries, [Hq, Hq + Hkv) keys,
// [Hq + Hkv, Hq + 2 Hkv) values (copied to the cache unchanged).  A null norm
// weight skips that norm (models without QK norms).
template <int D>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(const uint16_t* __restrict__ qkv,
                                                           const uint16_t* __restrict__ q_norm,
                                                           const uint16_t* __restrict__ k_norm, float eps,
                                                           const int32_t* __restrict__ depth, int P, double theta,
                                                           int Hq, int Hkv, uint16_t* __restrict__ q_out,
                                                           uint16_t* __restrict__ k_cache,
                                                           uint16_t* __restrict__ v_cache, long long cap) {
  constexpr int HALF = D / 2;
  const int n = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nh = Hq + 2 * Hkv;
  const uint16_t* src = qkv + (size_t)n * nh * D;
  const long long row = (long long)P + n;  // node n's cache row
  const bool act = lane < HALF;
  float cs = 1.f, sn = 0.f;
  if (act) {
    const double ang = (double)(P + depth[n]) * pow(theta, -2.0 * (double)lane / (double)D);
    double sd, cd;
    sincos(ang, &sd, &cd);
    cs = (float)cd;
    sn = (float)sd;
  }
  for (int hh = wave; hh < nh; hh += 4) {
    const uint16_t* hr = src + (size_t)hh * D;
    if (hh >= Hq + Hkv) {
      const int g = hh - Hq - Hkv;
      uint16_t* dst = v_cache + ((size_t)g * cap + row) * D;
      if (act) {
        dst[lane] = hr[lane];
        dst[lane + HALF] = hr[lane + HALF];
      }
      continue;
    }
    const bool is_q = hh < Hq;
    float a = act ? bf16_bits_to_f32(hr[lane]) : 0.f;
    float b = act ? bf16_bits_to_f32(hr[lane + HALF]) : 0.f;
    const uint16_t* nw = is_q ? q_norm : k_norm;
    if (nw) {
      float ss = __builtin_fmaf(a, a, b * b);
      for (int off = 32; off > 0; off >>= 1) ss += shfl_xor_f(ss, off);
      const float r = 1.f / sqrtf(ss / (float)D + eps);
      if (act) {
        a = a * r * bf16_bits_to_f32(nw[lane]);
        b = b * r * bf16_bits_to_f32(nw[lane + HALF]);
      }
    }
    const float ra = a * cs - b * sn, rb = b * cs + a * sn;
    uint16_t* dst = is_q ? q_out + ((size_t)n * Hq + hh) * D : k_cache + ((size_t)(hh - Hq) * cap + row) * D;
    if (act) {
      dst[lane] = f32_to_bf16_bits(ra);
      dst[lane + HALF] = f32_to_bf16_bits(rb);
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
  rmsnorm_kernel<<<n_rows, 256, 0, reinterpret_cast<hipStream_t>(stream)>>>(h, (const uint16_t*)weight, dim, eps,
                                                                           (uint16_t*)out);
  const hipError_t e = hipGetLastError();
  OOO_REQUIRE(e == hipSuccess, OOO_ERR_HIP, "ooo_rmsnorm: launch failed: %s", hipGetErrorString(e));
  return ooo::ok();
}

extern "C" int ooo_qk_norm_rope(const void* qkv, const void* q_norm, const void* k_norm, float eps,
                                const int32_t* depth, int32_t n_nodes, int32_t prefix_len, double rope_theta,
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
  if (head_dim == 128)
    qk_norm_rope_kernel<128><<<n_nodes, 256, 0, st>>>((const uint16_t*)qkv, (const uint16_t*)q_norm,
                                                      (const uint16_t*)k_norm, eps, depth, prefix_len, rope_theta,
                                                      n_q_heads, n_kv_heads, (uint16_t*)q_out, (uint16_t*)k_cache,
                                                      (uint16_t*)v_cache, cap);
  else
    qk_norm_rope_kernel<64><<<n_nodes, 256, 0, st>>>((const uint16_t*)qkv, (const uint16_t*)q_norm,
                                                     (const uint16_t*)k_norm, eps, depth, prefix_len, rope_theta,
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
