// Rotary position and per-head norm shared by the rotation kernels: the
// target's rotate-half RoPE at position P + depth of a trie node, after the
// per-head RMSNorm of q and k (Qwen3).
#pragma once

#include <math.h>

#include "device_common.h"

namespace ooo {

// Rotation frequencies theta^(-2j/D), j < D/2, computed on the host in double.
struct RopeFreq {
  double f[64];
};

inline RopeFreq rope_freq(double theta, int head_dim) {
  RopeFreq fr{};
  for (int j = 0; j < head_dim / 2; ++j) fr.f[j] = pow(theta, -2.0 * j / head_dim);
  return fr;
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float v) {
  return (uint16_t)(pack_bf16x2(v, 0.f) & 0xFFFFu);
}

// sin and cos of pos * f: the angle in double, reduced by multiples of 2 pi
// (two-term constant), so that a float sine/cosine of a small argument
// finishes it.
__device__ __forceinline__ void rope_sincos(int pos, double f, float& sn, float& cs) {
  const double ang = (double)pos * f;
  const double k = rint(ang * 0.15915494309189535);
  const double red = fma(-k, 2.4492935982947064e-16, fma(-k, 6.283185307179586, ang));
  sincosf((float)red, &sn, &cs);
}

// Lanes j < D/2 (act) hold the rotate-half pair (a, b) = (x[j], x[j + D/2])
// of one head; every lane of the wave calls this (the norm's sum of squares
// is a wave reduction).  Optional RMSNorm with weight nw (null: none), then
// the rotation by the angle whose sine and cosine are sn, cs.
__device__ __forceinline__ void norm_rotate(float& a, float& b, bool act, const uint16_t* nw, float eps, int D,
                                            int lane, float cs, float sn) {
  if (nw) {
    float ss = __builtin_fmaf(a, a, b * b);
    for (int off = 32; off > 0; off >>= 1) ss += shfl_xor_f(ss, off);
    const float r = 1.f / sqrtf(ss / (float)D + eps);
    if (act) {
      a = a * r * bf16_bits_to_f32(nw[lane]);
      b = b * r * bf16_bits_to_f32(nw[lane + D / 2]);
    }
  }
  const float ra = a * cs - b * sn, rb = b * cs + a * sn;
  a = ra;
  b = rb;
}

}  // namespace ooo
