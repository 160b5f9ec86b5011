// Device helpers shared by the forward and backward edge kernels:
// edge geometry, envelope, harmonics and the quintic radial table.
#pragma once

#include <hip/hip_runtime.h>

#include "common.h"

namespace dpa4c {

__device__ inline int lane_of() { return threadIdx.x & (kWave - 1); }

// A value that is the same in every lane of the wave, moved to a scalar
// register (out of the vector register budget).
__device__ inline float wave_uniform(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}

// Orders the LDS accesses of a wavefront: what its lanes wrote before is
// visible to its lanes after.  The fences cover LDS only, so outstanding
// global loads and stores of the wave are not waited for.
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Eq. (edge-geometry) in float32: rho = sqrt(|r|^2 + eps^2) and u = r / rho
// from one hardware reciprocal square root (v_rsq_f32, about 1 ulp; the
// argument is at least eps^2 = 1e-14, far from denormals).
struct EdgeGeom {
  float rho, ux, uy, uz, inv_rho;
};
__device__ inline EdgeGeom edge_geom(float rx, float ry, float rz) {
  EdgeGeom g;
  const float r2 = rx * rx + ry * ry + rz * rz + float(kEps * kEps);
  g.inv_rho = __builtin_amdgcn_rsqf(r2);
  g.rho = r2 * g.inv_rho;
  g.ux = rx * g.inv_rho;
  g.uy = ry * g.inv_rho;
  g.uz = rz * g.inv_rho;
  return g;
}

// Eq. (envelope): chi = t^4 (1 + 4x + 10x^2 + 20x^3 + 35x^4), x = rho/r_c,
// t = 1 - x, clipped; d chi / d rho = -280 x^4 t^3 / r_c.
__device__ inline void envelope(float rho, float inv_rc, float* chi, float* dchi) {
  float x = fminf(rho * inv_rc, 1.0f);
  float t = 1.0f - x;
  float t2 = t * t;
  float p = 1.0f + x * (4.0f + x * (10.0f + x * (20.0f + x * 35.0f)));
  *chi = t2 * t2 * p;
  if (dchi) {
    float x2 = x * x;
    *dchi = -280.0f * x2 * x2 * t2 * t * inv_rc;
  }
}

// Real Cartesian harmonics with |u|^2 set to one (Methods "Fidelity of the
// compressed model"; the error is O(eps^2/rho^2)).
__device__ inline void harm2(float x, float y, float z, float* b) {
  const float r3 = 1.7320508075688772f;
  b[0] = r3 * x * y;
  b[1] = r3 * y * z;
  b[2] = 0.5f * (3.0f * z * z - 1.0f);
  b[3] = r3 * x * z;
  b[4] = 0.5f * r3 * (x * x - y * y);
}
__device__ inline void harm3(float x, float y, float z, float* b) {
  const float a = 0.7905694150420949f;   // sqrt(5/8)
  const float r15 = 3.872983346207417f;  // sqrt(15)
  const float c = 0.6123724356957945f;   // sqrt(3/8)
  b[0] = a * y * (3.0f * x * x - y * y);
  b[1] = r15 * x * y * z;
  b[2] = c * y * (5.0f * z * z - 1.0f);
  b[3] = 0.5f * z * (5.0f * z * z - 3.0f);
  b[4] = c * x * (5.0f * z * z - 1.0f);
  b[5] = 0.5f * r15 * z * (x * x - y * y);
  b[6] = a * x * (x * x - 3.0f * y * y);
}
// gradients d B / d u (with |u|^2 = 1 held constant): g[m][3]
__device__ inline void harm2_grad(float x, float y, float z, float (*g)[3]) {
  const float r3 = 1.7320508075688772f;
  g[0][0] = r3 * y; g[0][1] = r3 * x; g[0][2] = 0.0f;
  g[1][0] = 0.0f;   g[1][1] = r3 * z; g[1][2] = r3 * y;
  g[2][0] = 0.0f;   g[2][1] = 0.0f;   g[2][2] = 3.0f * z;
  g[3][0] = r3 * z; g[3][1] = 0.0f;   g[3][2] = r3 * x;
  g[4][0] = r3 * x; g[4][1] = -r3 * y; g[4][2] = 0.0f;
}
__device__ inline void harm3_grad(float x, float y, float z, float (*g)[3]) {
  const float a = 0.7905694150420949f, r15 = 3.872983346207417f, c = 0.6123724356957945f;
  const float d = 0.5f * r15;
  g[0][0] = 6.0f * a * x * y;            g[0][1] = 3.0f * a * (x * x - y * y); g[0][2] = 0.0f;
  g[1][0] = r15 * y * z;                 g[1][1] = r15 * x * z;                g[1][2] = r15 * x * y;
  g[2][0] = 0.0f;                        g[2][1] = c * (5.0f * z * z - 1.0f);  g[2][2] = 10.0f * c * y * z;
  g[3][0] = 0.0f;                        g[3][1] = 0.0f;                       g[3][2] = 7.5f * z * z - 1.5f;
  g[4][0] = c * (5.0f * z * z - 1.0f);   g[4][1] = 0.0f;                       g[4][2] = 10.0f * c * x * z;
  g[5][0] = 2.0f * d * x * z;            g[5][1] = -2.0f * d * y * z;          g[5][2] = d * (x * x - y * y);
  g[6][0] = 3.0f * a * (x * x - y * y);  g[6][1] = -6.0f * a * x * y;          g[6][2] = 0.0f;
}

// Table interval and local coordinate tau in [0, 1) for rho.
// The row index is clamped to the table (a NaN rho maps to row 0 and gives
// a NaN tau, never an out-of-range read); beyond the last knot the last
// polynomial is extrapolated, where the envelope is already zero.
__device__ inline int table_row(float rho, float inv_delta, int n_rows, float* tau) {
  float s = rho * inv_delta;
  float sc = fminf(fmaxf(s, 0.0f), static_cast<float>(n_rows - 1));
  int r = static_cast<int>(sc);
  *tau = s - static_cast<float>(r);
  return r;
}

// Sum over aligned groups of G = 4, 8 or 16 lanes with DPP row permutations
// (quad xor 1, quad xor 2, half-row mirror, row mirror).  Every lane of the
// group ends with the same bits: each step adds a value and its partner, in
// the same order on both sides of the pair.
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int G>
__device__ inline float group_sum(float v) {
  static_assert(G == 4 || G == 8 || G == 16, "group of 4, 8 or 16 lanes");
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  if constexpr (G >= 8) v += dpp_f<0x141>(v);
  if constexpr (G == 16) v += dpp_f<0x140>(v);
  return v;
}

// Degree-two and degree-three harmonics as homogeneous polynomials of u
// (|u|^2 kept as x^2 + y^2 + z^2), Eq. (harmonics) and the degree-three
// block of the Supplementary Note.
__device__ inline void harm2_h(float x, float y, float z, float* b) {
  const float r3 = 1.7320508075688772f;
  b[0] = r3 * x * y;
  b[1] = r3 * y * z;
  b[2] = z * z - 0.5f * (x * x + y * y);
  b[3] = r3 * x * z;
  b[4] = 0.5f * r3 * (x * x - y * y);
}
__device__ inline void harm3_h(float x, float y, float z, float* b) {
  const float a = 0.7905694150420949f;   // sqrt(5/8)
  const float r15 = 3.872983346207417f;  // sqrt(15)
  const float c = 0.6123724356957945f;   // sqrt(3/8)
  const float x2 = x * x, y2 = y * y, z2 = z * z;
  b[0] = a * y * (3.0f * x2 - y2);
  b[1] = r15 * x * y * z;
  b[2] = c * y * (4.0f * z2 - x2 - y2);
  b[3] = z * (z2 - 1.5f * (x2 + y2));
  b[4] = c * x * (4.0f * z2 - x2 - y2);
  b[5] = 0.5f * r15 * z * (x2 - y2);
  b[6] = a * x * (x2 - 3.0f * y2);
}

// For weights w_m, sum_m w_m B_2m(u) = u.W u with the symmetric W below;
// returns M = 2W as (xx, yy, zz, xy, yz, xz), so that grad = M u.
__device__ inline void quad_form2(const float* w, float* M) {
  const float h3 = 0.8660254037844386f;   // sqrt(3)/2
  M[0] = 2.0f * (-0.5f * w[2] + h3 * w[4]);
  M[1] = 2.0f * (-0.5f * w[2] - h3 * w[4]);
  M[2] = 2.0f * w[2];
  M[3] = 2.0f * h3 * w[0];
  M[4] = 2.0f * h3 * w[1];
  M[5] = 2.0f * h3 * w[3];
}
// For weights w_m, P(u) = sum_m w_m B_3m(u) is a cubic in (x, y, z); G holds
// the coefficients of its gradient over the monomials (x^2, xy, xz, y^2, yz,
// z^2): dP/du_a = sum_q G[a][q] mono_q.  P = u . grad P / 3.
__device__ inline void cubic_form3(const float* w, float (*G)[6]) {
  const float a = 0.7905694150420949f, b = 3.872983346207417f, c = 0.6123724356957945f;
  const float d = 0.5f * b;
  const float pxxx = -c * w[4] + a * w[6];
  const float pxxy = 3.0f * a * w[0] - c * w[2];
  const float pxxz = -1.5f * w[3] + d * w[5];
  const float pxyy = -c * w[4] - 3.0f * a * w[6];
  const float pxyz = b * w[1];
  const float pxzz = 4.0f * c * w[4];
  const float pyyy = -a * w[0] - c * w[2];
  const float pyyz = -1.5f * w[3] - d * w[5];
  const float pyzz = 4.0f * c * w[2];
  const float pzzz = w[3];
  G[0][0] = 3.0f * pxxx; G[0][1] = 2.0f * pxxy; G[0][2] = 2.0f * pxxz;
  G[0][3] = pxyy;        G[0][4] = pxyz;        G[0][5] = pxzz;
  G[1][0] = pxxy;        G[1][1] = 2.0f * pxyy; G[1][2] = pxyz;
  G[1][3] = 3.0f * pyyy; G[1][4] = 2.0f * pyyz; G[1][5] = pyzz;
  G[2][0] = pxxz;        G[2][1] = pxyz;        G[2][2] = 2.0f * pxzz;
  G[2][3] = pyyz;        G[2][4] = 2.0f * pyzz; G[2][5] = 3.0f * pzzz;
}

// Degree four (Supplementary Note, real solid harmonics of degrees three and
// four), as homogeneous quartics in (x, y, z), so exact off the unit sphere.
__device__ inline void harm4_h(float x, float y, float z, float* b) {
  const float x2 = x * x, y2 = y * y, z2 = z * z;
  const float h35 = 2.958039891549808f;    // sqrt(35)/2
  const float q70 = 2.091650066335189f;    // sqrt(70)/4
  const float h5 = 1.118033988749895f;     // sqrt(5)/2
  const float q10 = 0.7905694150420949f;   // sqrt(10)/4
  const float q5 = 0.5590169943749475f;    // sqrt(5)/4
  const float e35 = 0.739509972887452f;    // sqrt(35)/8
  b[0] = h35 * x * y * (x2 - y2);
  b[1] = q70 * y * z * (3.0f * x2 - y2);
  b[2] = h5 * x * y * (6.0f * z2 - x2 - y2);
  b[3] = q10 * y * z * (4.0f * z2 - 3.0f * x2 - 3.0f * y2);
  b[4] = 0.375f * (x2 * x2 + y2 * y2) + z2 * z2 + 0.75f * x2 * y2 - 3.0f * z2 * (x2 + y2);
  b[5] = q10 * x * z * (4.0f * z2 - 3.0f * x2 - 3.0f * y2);
  b[6] = q5 * (x2 - y2) * (6.0f * z2 - x2 - y2);
  b[7] = q70 * x * z * (x2 - 3.0f * y2);
  b[8] = e35 * (x2 * x2 - 6.0f * x2 * y2 + y2 * y2);
}

// Monomial coefficients p[15] of P(u) = sum_m w_m B_4m(u) over the quartic
// monomials x^a y^b z^c (a+b+c = 4) in the order index(a, c) =
// (4-a)(5-a)/2 + c: x^4, x^3y, x^3z, x^2y^2, x^2yz, x^2z^2, xy^3, xy^2z,
// xyz^2, xz^3, y^4, y^3z, y^2z^2, yz^3, z^4.
__device__ inline void quartic_coeffs4(const float* w, float* p) {
  const float h35 = 2.958039891549808f, q70 = 2.091650066335189f, h5 = 1.118033988749895f;
  const float r10 = 3.1622776601683795f, q5 = 0.5590169943749475f, e35 = 0.739509972887452f;
  const float t10 = 0.75f * r10, t70 = 3.0f * q70;   // 3 sqrt(10)/4, 3 sqrt(70)/4
  p[0] = 0.375f * w[4] - q5 * w[6] + e35 * w[8];
  p[1] = h35 * w[0] - h5 * w[2];
  p[2] = -t10 * w[5] + q70 * w[7];
  p[3] = 0.75f * w[4] - 6.0f * e35 * w[8];
  p[4] = t70 * w[1] - t10 * w[3];
  p[5] = -3.0f * w[4] + 6.0f * q5 * w[6];
  p[6] = -h35 * w[0] - h5 * w[2];
  p[7] = -t10 * w[5] - t70 * w[7];
  p[8] = 6.0f * h5 * w[2];
  p[9] = r10 * w[5];
  p[10] = 0.375f * w[4] + q5 * w[6] + e35 * w[8];
  p[11] = -q70 * w[1] - t10 * w[3];
  p[12] = -3.0f * w[4] - 6.0f * q5 * w[6];
  p[13] = r10 * w[3];
  p[14] = w[4];
}

// Gradient of the quartic with monomial coefficients p[15]: dP/du_d =
// sum_q G[d][q] mono3_q over the cubic monomials in the order index(a, c) =
// (3-a)(4-a)/2 + c: x^3, x^2y, x^2z, xy^2, xyz, xz^2, y^3, y^2z, yz^2, z^3.
// P = u . grad P / 4.
__device__ inline void quartic_grad4(const float* p, float (*G)[10]) {
#pragma unroll
  for (int d = 0; d < 3; ++d)
#pragma unroll
    for (int q = 0; q < 10; ++q) G[d][q] = 0.0f;
#pragma unroll
  for (int a = 4; a >= 0; --a)
#pragma unroll
    for (int c = 0; c <= 4 - a; ++c) {
      const int b = 4 - a - c;
      const float v = p[(4 - a) * (5 - a) / 2 + c];
      if (a > 0) G[0][(4 - a) * (5 - a) / 2 + c] += float(a) * v;       // x^(a-1) y^b z^c
      if (b > 0) G[1][(3 - a) * (4 - a) / 2 + c] += float(b) * v;       // x^a y^(b-1) z^c
      if (c > 0) G[2][(3 - a) * (4 - a) / 2 + c - 1] += float(c) * v;   // x^a y^b z^(c-1)
    }
}

// the ten cubic monomials of quartic_grad4's order
__device__ inline void cubic_monomials(float x, float y, float z, float* m) {
  const float x2 = x * x, y2 = y * y, z2 = z * z;
  m[0] = x2 * x; m[1] = x2 * y; m[2] = x2 * z; m[3] = x * y2; m[4] = x * y * z;
  m[5] = x * z2; m[6] = y2 * y; m[7] = y2 * z; m[8] = y * z2; m[9] = z2 * z;
}

// species index clamped into the type table (the padding type for bad input)
__device__ inline int clamp_type(int a, int n_types1) {
  return static_cast<unsigned>(a) < static_cast<unsigned>(n_types1) ? a : n_types1 - 1;
}

// quintic in normalised form: value (Horner)
__device__ inline float quintic_val(const float* c, float t) {
  return c[0] + t * (c[1] + t * (c[2] + t * (c[3] + t * (c[4] + t * c[5]))));
}

// load 6 floats from an 8-byte aligned address as three float2
__device__ inline void load6(const float* __restrict__ p, float* c) {
  const float2* q = reinterpret_cast<const float2*>(p);
  float2 a = q[0], b = q[1], d = q[2];
  c[0] = a.x; c[1] = a.y; c[2] = b.x; c[3] = b.y; c[4] = d.x; c[5] = d.y;
}

// lane 0 of every group of W lanes to all lanes of its group
template <int W>
__device__ inline float4 group_bcast(float4 v) {
  v.x = __shfl(v.x, 0, W);
  v.y = __shfl(v.y, 0, W);
  v.z = __shfl(v.z, 0, W);
  v.w = __shfl(v.w, 0, W);
  return v;
}

// The lane's entries of a folded table row (kFoldWords * C0 words) for its
// CPL channels c = k + LPE j.  The row holds first the (c0, c1) float32 pairs
// and then the words of scaled float16 (c2, c3), each permuted so that a
// lane's values are adjacent: the pairs of its channels j = 2q, 2q + 1 form
// the 16 bytes at (q LPE + k) * 4, and the words of j = 4q .. 4q + 3 the 16
// bytes at 2 C0 + (q LPE + k) * 4 (8 bytes at 2 C0 + 2 k when CPL = 2).  A
// lane thus reads its 12 CPL bytes with 16-byte loads, the group at unit
// stride.  T[j] = (c0, c1, word) of channel j.
template <int LPE, int CPL>
__device__ inline void load_fold_row(const float* __restrict__ row, int k, float3* T) {
  static_assert(CPL == 2 || CPL % 4 == 0, "folded row layout");
  float4 a[CPL / 2];
#pragma unroll
  for (int q = 0; q < CPL / 2; ++q) a[q] = *reinterpret_cast<const float4*>(row + (q * LPE + k) * 4);
  uint32_t w[CPL];
  const float* wrow = row + 2 * LPE * CPL;
  if constexpr (CPL == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(wrow + 2 * k);
    w[0] = v.x;
    w[1] = v.y;
  } else {
#pragma unroll
    for (int q = 0; q < CPL / 4; ++q) {
      const uint4 v = *reinterpret_cast<const uint4*>(wrow + (q * LPE + k) * 4);
      w[4 * q] = v.x;
      w[4 * q + 1] = v.y;
      w[4 * q + 2] = v.z;
      w[4 * q + 3] = v.w;
    }
  }
#pragma unroll
  for (int j = 0; j < CPL; ++j) {
    const float4& p = a[j / 2];
    T[j] = (j & 1) ? make_float3(p.z, p.w, __uint_as_float(w[j]))
                   : make_float3(p.x, p.y, __uint_as_float(w[j]));
  }
}
__device__ inline float half_lo(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h & 0xFFFFu)));
}
__device__ inline float half_hi(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h >> 16)));
}

}  // namespace dpa4c
