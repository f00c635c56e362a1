// RoPE arithmetic shared by the kernels that rotate keys (internal, not part of the C ABI):
// the fp64 angle of a feature pair, the compensated fp32 rotation and 16-byte key packs.
#pragma once

#include "device_common.h"

#include <cmath>

namespace nexus {

constexpr double kTwoPiHi = 6.283185307179586232;       // fp64(2*pi)
constexpr double kTwoPiLo = 2.4492935982947064e-16;     // 2*pi - fp64(2*pi)
constexpr int kMaxPairs = 512;                            // head_dim <= 1024

// cos and sin of delta * theta_i, theta_i = base^(-2i/D): the angle is formed and reduced
// modulo 2 pi in fp64 (two-term 2 pi), then sincos in fp64.
__device__ __forceinline__ void pair_angle(int64_t delta, double base, int i, int head_dim,
                                           double &c, double &s) {
  const double theta = pow(base, -2.0 * (double)i / (double)head_dim);
  const double ang = (double)delta * theta;
  const double k = rint(ang / kTwoPiHi);
  double r = fma(-k, kTwoPiHi, ang);
  r = fma(-k, kTwoPiLo, r);
  sincos(r, &s, &c);
}

template <typename T>
struct Pack;  // 16 bytes of keys

template <>
struct Pack<uint16_t> {  // 8 bf16
  static constexpr int N = 8;
  __device__ static void unpack(const u32x4 &v, float *x) {
    const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[2 * e] = __uint_as_float(w[e] << 16);
      x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  }
  __device__ static u32x4 pack(const float *x) {
    return u32x4{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                 pack_bf16x2(x[6], x[7])};
  }
};

template <>
struct Pack<uint32_t> {  // 4 f32
  static constexpr int N = 4;
  __device__ static void unpack(const u32x4 &v, float *x) {
    x[0] = __uint_as_float(v[0]);
    x[1] = __uint_as_float(v[1]);
    x[2] = __uint_as_float(v[2]);
    x[3] = __uint_as_float(v[3]);
  }
  __device__ static u32x4 pack(const float *x) {
    return u32x4{__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                 __float_as_uint(x[3])};
  }
};

// u c - w s with c = ch + cl, s = sh + sl: w sh = p + e exactly (two-product by FMA), then
// (u ch - p) rounded once by an FMA, plus the small terms (u cl - w sl) - e.
__device__ __forceinline__ float rot_dot(float u, float w, float ch, float cl, float sh, float sl) {
  const float p = w * sh;
  const float e = fmaf(w, sh, -p);
  const float r = fmaf(u, ch, -p);
  const float t = fmaf(u, cl, -(w * sl));
  return r + (t - e);
}

// Rotate pairs (a[e], b[e]) by the angle whose cos/sin head and tail are (ch, cl, sh, sl)[e].
template <int N>
__device__ __forceinline__ void rotate(float *a, float *b, const float *ch, const float *cl,
                                       const float *sh, const float *sl) {
#pragma unroll
  for (int e = 0; e < N; ++e) {
    const float xa = a[e], xb = b[e];
    a[e] = rot_dot(xa, xb, ch[e], cl[e], sh[e], sl[e]);      // xa c - xb s
    b[e] = rot_dot(xb, -xa, ch[e], cl[e], sh[e], sl[e]);     // xb c + xa s
  }
}

// cos / sin head and tail of every pair of one rotation (angle delta * theta_i for all rows),
// formed on the host by the same steps as pair_angle / pair_cs and passed to a kernel by value:
// the fp64 angle code then stays out of the kernel (with it, the re-anchor needs 117 registers
// and its workgroups spend their start on the angles; without, 68).
constexpr int kTabPairs = 128;   // head_dim <= 256
struct RopeTab {
  float v[4][kTabPairs];         // cos head, cos tail, sin head, sin tail
};
inline void rope_tab_host(int64_t delta, double base, int head_dim, RopeTab &t) {
  for (int i = 0; i < head_dim / 2 && i < kTabPairs; ++i) {
    const double theta = std::pow(base, -2.0 * (double)i / (double)head_dim);
    const double ang = (double)delta * theta;
    const double k = std::rint(ang / kTwoPiHi);
    double r = std::fma(-k, kTwoPiHi, ang);
    r = std::fma(-k, kTwoPiLo, r);
    const double c = std::cos(r), s = std::sin(r);
    t.v[0][i] = (float)c;
    t.v[1][i] = (float)(c - (double)t.v[0][i]);
    t.v[2][i] = (float)s;
    t.v[3][i] = (float)(s - (double)t.v[2][i]);
  }
}

// fp32 head + tail of the cosine and sine of pair i at angle delta * theta_i
__device__ __forceinline__ void pair_cs(int64_t delta, double base, int i, int head_dim,
                                        float &ch, float &cl, float &sh, float &sl) {
  double c, s;
  pair_angle(delta, base, i, head_dim, c, s);
  ch = (float)c;
  cl = (float)(c - (double)ch);
  sh = (float)s;
  sl = (float)(s - (double)sh);
}

}  // namespace nexus
