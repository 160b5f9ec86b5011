// Per-atom invariant readout (Methods "Nonlinear readout and atomic energy",
// Eqs. (alignment) .. (calibration)) and its vector-Jacobian product.  Half a
// wavefront (32 lanes) serves one atom, so a wave reads out two atoms side by
// side; each atom has its own LDS block, and the descriptor row (D~, D or
// dE/dD) lives in a caller-provided LDS row.
//
// Each stage spreads its outputs over the lanes (gather form: every output is
// computed by one lane from values written by the previous stage), so the
// results do not depend on scheduling.  The (1,1,2) and (2,2,2) bispectrum
// blocks use the closed forms of Eq. (closed-forms); (1,2,3) and (2,3,3)
// contract the dense coupling tensors one index at a time:
//   J123[k1][k2] = sum_m1 Z1[m1][k1] U[m1][k2],  U = T Z2,  T[m1][m2] = sum_m3 C123 Z3
//   J233[e]      = sum_m1 Z2[m1][e] V[m1],       V = W Z3,  W[m1][m2] = sum_m3 C233 Z3
// The couplings (C123 [3][5][7] then C233 [5][7][7], the latter symmetric in
// its last two indices) and the other readout parameters are read from a
// ReadoutParams block staged in LDS by the caller.  The two entry points are
// not inlined: they get their own register allocation instead of adding to
// the pressure of the MLP code around their call sites.  Their LDS arguments
// carry the LDS address space, so every access is a ds_read / ds_write.
#pragma once

#include "common.h"
#include "edge_math.h"

namespace dpa4c {

#define DPA4C_LDS __attribute__((address_space(3)))

constexpr int kHalf = 32;   // lanes per atom

// sum_q a[q] b[q] over N (a multiple of 4) values of two 16-byte aligned LDS
// rows, four at a time
typedef float lds_f4 __attribute__((ext_vector_type(4)));
template <int N>
__device__ inline float lds_dot(const DPA4C_LDS float* a, const DPA4C_LDS float* b) {
  static_assert(N % 4 == 0, "rows of whole 16-byte vectors");
  float acc = 0.0f;
#pragma unroll
  for (int q = 0; q < N / 4; ++q) {
    const lds_f4 x = *reinterpret_cast<const DPA4C_LDS lds_f4*>(a + 4 * q);
    const lds_f4 y = *reinterpret_cast<const DPA4C_LDS lds_f4*>(b + 4 * q);
    acc = fmaf(x.x, y.x, acc);
    acc = fmaf(x.y, y.y, acc);
    acc = fmaf(x.z, y.z, acc);
    acc = fmaf(x.w, y.w, acc);
  }
  return acc;
}

// vech index t -> (c, c') with c <= c', row-major over the upper triangle
__device__ inline void vech_pair(int t, int C, int* c, int* cp) {
  int r = 0;
  while (t >= C - r) {
    t -= C - r;
    ++r;
  }
  *c = r;
  *cp = r + t;
}

// Readout parameters staged once per workgroup into LDS (the readout reads
// each of them many times per atom).
// The matrices are also kept transposed (W1T[c'][c] = W1[c][c'], ...) so that
// both the products and their adjoints read contiguous 16-byte rows.
template <class P>
struct ReadoutParams {
  alignas(16) float W1[P::C1 * P::C1];     // alignment, degree 1 (I + W applied in-kernel)
  alignas(16) float W2[P::C2 * P::C2];
  alignas(16) float A1[P::kHasA1 ? P::C1 * P::K1 : 1]; // probes, degree 1 (identity when K1 = C1)
  alignas(16) float A2[P::C2 * P::K2];
  alignas(16) float W1T[P::C1 * P::C1];
  alignas(16) float W2T[P::C2 * P::C2];
  alignas(16) float A1T[P::kHasA1 ? P::C1 * P::K1 : 1];
  alignas(16) float A2T[P::C2 * P::K2];
  float mu[P::DSTR];                       // calibration, zero padded
  float inv_sigma[P::DSTR];
  float cpl[P::L >= 3 ? couplings_for(P::L) : 1];   // C123, C233 (then the degree-four ones)
  // (c, c') of every vech index, c | c' << 8: degree one (C1) and degree two
  // (C2, which is also K1)
  uint16_t vp1[P::nG1];
  uint16_t vp2[P::nG2];
};

// Cooperative copy of the readout parameters by the ``nthreads`` threads of
// a workgroup; the caller synchronises afterwards.
template <class P>
__device__ void stage_readout_params(ReadoutParams<P>& rp, const ModelDev& md, int tid,
                                     int nthreads) {
  for (int t = tid; t < P::C1 * P::C1; t += nthreads) {
    rp.W1[t] = md.W1[t];
    rp.W1T[(t % P::C1) * P::C1 + t / P::C1] = md.W1[t];
  }
  for (int t = tid; t < P::C2 * P::C2; t += nthreads) {
    rp.W2[t] = md.W2[t];
    rp.W2T[(t % P::C2) * P::C2 + t / P::C2] = md.W2[t];
  }
  if constexpr (P::kHasA1)
    for (int t = tid; t < P::C1 * P::K1; t += nthreads) {
      rp.A1[t] = md.A1[t];
      rp.A1T[(t % P::K1) * P::C1 + t / P::K1] = md.A1[t];
    }
  for (int t = tid; t < P::C2 * P::K2; t += nthreads) {
    rp.A2[t] = md.A2[t];
    rp.A2T[(t % P::K2) * P::C2 + t / P::K2] = md.A2[t];
  }
  for (int t = tid; t < P::DSTR; t += nthreads) {
    rp.mu[t] = t < P::DOUT ? md.mu[t] : 0.0f;
    rp.inv_sigma[t] = t < P::DOUT ? md.inv_sigma[t] : 0.0f;
  }
  if constexpr (P::L >= 3)
    for (int t = tid; t < couplings_for(P::L); t += nthreads) rp.cpl[t] = md.cpl[t];
  for (int t = tid; t < P::nG1 + P::nG2; t += nthreads) {
    const bool one = t < P::nG1;
    int c, cp;
    vech_pair(one ? t : t - P::nG1, one ? P::C1 : P::C2, &c, &cp);
    (one ? rp.vp1[t] : rp.vp2[t - P::nG1]) = static_cast<uint16_t>(c | (cp << 8));
  }
}

// Rows that are read as 16-byte vectors are 16-byte aligned: the node state
// starts 8 bytes into the (aligned) block, so that its Y blocks are.
template <class P>
struct alignas(16) ReadoutLds {
  float ypad_[2];
  float y[P::NS];                 // [S0, S1, Y]
  alignas(16) float xt1[3 * P::C1];   // aligned features, Eq. (alignment)
  alignas(16) float xt2[5 * P::C2];
  float xt3[8];                   // degree three (identity probe: Z3 = X~3)
  alignas(16) float z1[3 * P::K1];    // probes, Eq. (probes)
  // channel-major copies, the degree index padded with zeros to 4 (8):
  // xt1c[c][m] = xt1[m][c], xt2c[c][m] = xt2[m][c], z1c[k][a] = z1[a][k]
  alignas(16) float xt1c[P::C1 * 4];
  alignas(16) float xt2c[P::C2 * 8];
  alignas(16) float z1c[P::K1 * 4];
  float z2[5 * P::K2];
  float q[P::K2][9];              // STF matrices of the degree-two probes
  alignas(16) float qv[P::K2][P::K1][4];   // Q_eta v_kappa (fourth entry zero)
  float t123[15], u123[3 * P::K2], w233[35], v233[5];
  // degree four (one channel; Z4 = X~4): X~4, T134[m1] = C134 : Z3 Z4,
  // T224[m1][m2] = C224 . Z4, T244[m1] = C244 : Z4 Z4
  float xt4[P::L >= 4 ? 9 : 1], t134[P::L >= 4 ? 3 : 1], t224[P::L >= 4 ? 25 : 1],
      t244[P::L >= 4 ? 5 : 1];
  // backward only
  alignas(16) float gxt1[3 * P::C1];
  alignas(16) float gxt2[5 * P::C2];
  // the Gram adjoints as full symmetric matrices, weights included:
  // Gbar[c][c'] = dE/dG_cc' times 2 (c = c') or sqrt(2)
  alignas(16) float gb1[P::C1 * P::C1];
  alignas(16) float gb2[P::C2 * P::C2];
  float gxt3[8];
  alignas(16) float gz1[3 * P::K1];
  float gz2[5 * P::K2];
  float gz3[8];
  float gq[P::K2][9];
  float ub123[3 * P::K2], tb123[15], vb233[5];
  float gxt4[P::L >= 4 ? 9 : 1], tb134[P::L >= 4 ? 3 : 1], tb224[P::L >= 4 ? 25 : 1],
      tb244[P::L >= 4 ? 5 : 1];
  float gy[P::NS];
};

constexpr float kSqrt2 = 1.4142135623730951f;
constexpr float kInvSqrt2 = 0.7071067811865476f;
constexpr float kInvSqrt6 = 0.4082482904638631f;
constexpr float kInvSqrt5 = 0.4472135954999579f;
constexpr float kSqrt12_35 = 0.5855400437691199f;


// STF(z) of Eq. (stf) in the basis order (xy, yz, z^2, xz, x^2 - y^2):
// entry (a, b) of the symmetric trace-free matrix
template <class T>
__device__ inline float stf_entry(const T* z, int stride, int a, int b) {
  float z0 = z[0], z1 = z[stride], z2 = z[2 * stride], z3 = z[3 * stride], z4 = z[4 * stride];
  if (a > b) { int t = a; a = b; b = t; }
  if (a == 0 && b == 0) return -z2 * kInvSqrt6 + z4 * kInvSqrt2;
  if (a == 1 && b == 1) return -z2 * kInvSqrt6 - z4 * kInvSqrt2;
  if (a == 2 && b == 2) return 2.0f * z2 * kInvSqrt6;
  if (a == 0 && b == 1) return z0 * kInvSqrt2;
  if (a == 1 && b == 2) return z1 * kInvSqrt2;
  return z3 * kInvSqrt2;   // (0, 2)
}
// adjoint: dE/dz_m = E_m : Qbar for a (not necessarily symmetric) 3x3 Qbar
template <class T>
__device__ inline float stf_adjoint(const T* g, int m) {
  switch (m) {
    case 0: return (g[1] + g[3]) * kInvSqrt2;
    case 1: return (g[5] + g[7]) * kInvSqrt2;
    case 2: return (-g[0] - g[4] + 2.0f * g[8]) * kInvSqrt6;
    case 3: return (g[2] + g[6]) * kInvSqrt2;
    default: return (g[0] - g[4]) * kInvSqrt2;
  }
}

// index of the (k1 <= k2) pair in row-major order over the upper triangle
__device__ inline int tri_index(int k1, int k2, int K) { return k1 * K - k1 * (k1 - 1) / 2 + (k2 - k1); }

// the four (2,2,2) entries for K2 = 2: (0,0,0) (0,0,1) (0,1,1) (1,1,1)
__device__ inline void e222(int t, int* a, int* b, int* c, float* w) {
  const float r3 = 1.7320508075688772f;
  *a = t >= 3 ? 1 : 0;
  *b = t >= 2 ? 1 : 0;
  *c = t >= 1 ? 1 : 0;
  *w = (t == 0 || t == 3) ? 1.0f : r3;
}

// fixed-order sum over the 32 lanes of a half wave (butterfly; every lane of
// the half gets the same bits)
__device__ inline float half_sum(float v) {
  for (int off = 1; off < kHalf; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

// Forward intermediates from s.y: M, aligned features, probes, Q, Qv and the
// partial contractions T, U, W, V of the generic couplings.
template <class P>
__device__ inline void readout_intermediates(DPA4C_LDS ReadoutLds<P>& s,
                                             const DPA4C_LDS ReadoutParams<P>& rp, float* M0,
                                             float* M1) {
  const DPA4C_LDS float* cpl = rp.cpl;
  const int lane = lane_of() & (kHalf - 1);
  const float m0 = sqrtf(0.25f + s.y[0]);
  const float m1 = sqrtf(0.25f + s.y[1]);
  *M0 = m0;
  *M1 = m1;
  const float i1 = 1.0f / m1;
  constexpr int n1 = 3 * P::C1, n2 = 5 * P::C2, n3 = (P::L >= 3 ? 7 : 0);
  constexpr int n4 = (P::L >= 4 ? 9 : 0);
  for (int o = lane; o < n1 + n2 + n3 + n4; o += kHalf) {
    if (o < n1) {
      int m = o / P::C1, cp = o % P::C1;
      const DPA4C_LDS float* x = s.y + P::Y1 + m * P::C1;
      const float v = (x[cp] + lds_dot<P::C1>(x, rp.W1T + cp * P::C1)) * i1;
      s.xt1[o] = v;
      s.xt1c[cp * 4 + m] = v;
      if (m == 0) s.xt1c[cp * 4 + 3] = 0.0f;
    } else if (o < n1 + n2) {
      int t = o - n1, m = t / P::C2, cp = t % P::C2;
      const DPA4C_LDS float* x = s.y + P::Y2 + m * P::C2;
      const float v = (x[cp] + lds_dot<P::C2>(x, rp.W2T + cp * P::C2)) * i1;
      s.xt2[t] = v;
      s.xt2c[cp * 8 + m] = v;
      if (m == 0) s.xt2c[cp * 8 + 5] = s.xt2c[cp * 8 + 6] = s.xt2c[cp * 8 + 7] = 0.0f;
    } else if (o < n1 + n2 + n3) {
      int m = o - n1 - n2;
      s.xt3[m] = s.y[P::Y3 + m] * i1;
    } else if constexpr (P::L >= 4) {
      int m = o - n1 - n2 - n3;
      s.xt4[m] = s.y[P::Y4 + m] * i1;
    }
  }
  wave_sync();
  for (int o = lane; o < 3 * P::K1 + 5 * P::K2; o += kHalf) {
    if (o < 3 * P::K1) {
      int m = o / P::K1, k = o % P::K1;
      float acc;
      if constexpr (P::kHasA1) {
        acc = lds_dot<P::C1>(s.xt1 + m * P::C1, rp.A1T + k * P::C1);
      } else {
        acc = s.xt1[m * P::C1 + k];
      }
      s.z1[o] = acc;
      s.z1c[k * 4 + m] = acc;
      if (m == 0) s.z1c[k * 4 + 3] = 0.0f;
    } else {
      int t = o - 3 * P::K1, m = t / P::K2, k = t % P::K2;
      s.z2[t] = lds_dot<P::C2>(s.xt2 + m * P::C2, rp.A2T + k * P::C2);
    }
  }
  if constexpr (P::L >= 3) {
    // T[m1][m2] = sum_m3 C123 Z3 (15 entries), W[m1][m2] = sum_m3 C233 Z3 (35)
    for (int o = lane; o < 50; o += kHalf) {
      const DPA4C_LDS float* c = cpl + 7 * o;   // C233 follows C123 (15 rows of 7)
      float acc = 0.0f;
#pragma unroll
      for (int m3 = 0; m3 < 7; ++m3) acc += c[m3] * s.xt3[m3];
      if (o < 15) s.t123[o] = acc;
      else s.w233[o - 15] = acc;
    }
  }
  if constexpr (P::L >= 4) {
    // T134[m1] = sum C134[m1][m3][m4] Z3 Z4, T224[m1][m2] = sum_m4 C224 Z4,
    // T244[m1] = sum C244[m1][a][b] Z4 Z4 (33 entries, fixed order each)
    for (int o = lane; o < 33; o += kHalf) {
      float acc = 0.0f;
      if (o < 3) {
        const DPA4C_LDS float* c = cpl + kO134 + 63 * o;
#pragma unroll
        for (int m3 = 0; m3 < 7; ++m3) {
          float r = 0.0f;
#pragma unroll
          for (int m4 = 0; m4 < 9; ++m4) r += c[9 * m3 + m4] * s.xt4[m4];
          acc += r * s.xt3[m3];
        }
        s.t134[o] = acc;
      } else if (o < 28) {
        const DPA4C_LDS float* c = cpl + kO224 + 9 * (o - 3);
#pragma unroll
        for (int m4 = 0; m4 < 9; ++m4) acc += c[m4] * s.xt4[m4];
        s.t224[o - 3] = acc;
      } else {
        const DPA4C_LDS float* c = cpl + kO244 + 81 * (o - 28);
#pragma unroll
        for (int a = 0; a < 9; ++a) {
          float r = 0.0f;
#pragma unroll
          for (int b = 0; b < 9; ++b) r += c[9 * a + b] * s.xt4[b];
          acc += r * s.xt4[a];
        }
        s.t244[o - 28] = acc;
      }
    }
  }
  wave_sync();
  if (lane < P::K2 * 9) {
    int eta = lane / 9, ab = lane % 9;
    s.q[eta][ab] = stf_entry(s.z2 + eta, P::K2, ab / 3, ab % 3);
  }
  if constexpr (P::L >= 3) {
    // U[m1][k2] = sum_m2 T[m1][m2] Z2[m2][k2],  V[m1] = sum_m2 W[m1][m2] Z3[m2]
    static_assert(P::K2 * 9 <= 18 && 3 * P::K2 <= 6, "lane plan of the readout");
    if (lane >= 18 && lane < 18 + 3 * P::K2) {
      const int o = lane - 18, m1 = o / P::K2, k2 = o % P::K2;
      float acc = 0.0f;
#pragma unroll
      for (int m2 = 0; m2 < 5; ++m2) acc += s.t123[m1 * 5 + m2] * s.z2[m2 * P::K2 + k2];
      s.u123[o] = acc;
    } else if (lane >= 24 && lane < 29) {
      const int m1 = lane - 24;
      float acc = 0.0f;
#pragma unroll
      for (int m2 = 0; m2 < 7; ++m2) acc += s.w233[m1 * 7 + m2] * s.xt3[m2];
      s.v233[m1] = acc;
    }
  }
  wave_sync();
  for (int o = lane; o < P::K2 * P::K1 * 3; o += kHalf) {
    int eta = o / (P::K1 * 3), k = (o / 3) % P::K1, a = o % 3;
    float acc = 0.0f;
#pragma unroll
    for (int b = 0; b < 3; ++b) acc += s.q[eta][a * 3 + b] * s.z1[b * P::K1 + k];
    s.qv[eta][k][a] = acc;
    if (a == 0) s.qv[eta][k][3] = 0.0f;
  }
  wave_sync();
}

// Eqs. (gram) .. (calibration): writes the calibrated descriptor to the LDS
// row ``d`` (P::DSTR entries, zero padded).  s.y must hold the node state and
// ``x0`` is the atom's row of the type table (Eq. (init-features)).
template <class P>
__device__ __attribute__((noinline)) void readout_forward(DPA4C_LDS ReadoutLds<P>& s,
                                                          const DPA4C_LDS ReadoutParams<P>& rp,
                                                          const float* __restrict__ x0,
                                                          DPA4C_LDS float* d) {
  const int lane = lane_of() & (kHalf - 1);
  const DPA4C_LDS float* cpl = rp.cpl;
  // the atom's row of the type table, requested before the LDS work
  constexpr int NX = (P::C0 + kHalf - 1) / kHalf;
  float x0r[NX];
#pragma unroll
  for (int q = 0; q < NX; ++q) x0r[q] = lane + q * kHalf < P::C0 ? x0[lane + q * kHalf] : 0.0f;
  // every entry is calibrated (Eq. (calibration)) as it is written
  auto put = [&](int o, float v) { d[o] = (v - rp.mu[o]) * rp.inv_sigma[o]; };
  float M0, M1;
  readout_intermediates<P>(s, rp, &M0, &M1);
  const float i0 = 1.0f / M0;
#pragma unroll
  for (int q = 0; q < NX; ++q) {
    const int c = lane + q * kHalf;
    if (c < P::C0) {
      put(P::oX0 + c, x0r[q]);
      put(P::oX + c, s.y[P::Y0 + c] * i0);
    }
  }
  if (lane == 0) {
    put(P::oM0, M0);
    put(P::oM1, M1);
  }
  if (lane < P::DSTR - P::DOUT) d[P::DOUT + lane] = 0.0f;   // zero padding
  // Gram blocks, Eq. (gram), vech with sqrt(2) off the diagonal
  for (int o = lane; o < P::nG1 + P::nG2 + P::nG3 + P::nG4; o += kHalf) {
    float acc = 0.0f;
    if (o < P::nG1) {
      const int c = rp.vp1[o] & 0xFF, cp = rp.vp1[o] >> 8;
      acc = lds_dot<4>(s.xt1c + 4 * c, s.xt1c + 4 * cp);
      if (c != cp) acc *= kSqrt2;
    } else if (o < P::nG1 + P::nG2) {
      const int c = rp.vp2[o - P::nG1] & 0xFF, cp = rp.vp2[o - P::nG1] >> 8;
      acc = lds_dot<8>(s.xt2c + 8 * c, s.xt2c + 8 * cp);
      if (c != cp) acc *= kSqrt2;
    } else if (o < P::nG1 + P::nG2 + P::nG3) {
#pragma unroll
      for (int m = 0; m < 7; ++m) acc += s.xt3[m] * s.xt3[m];
    } else if constexpr (P::L >= 4) {
#pragma unroll
      for (int m = 0; m < 9; ++m) acc += s.xt4[m] * s.xt4[m];
    }
    put(P::oG1 + o, acc);
  }
  // (1,1,2): -(f/sqrt5) v_k1 . Q_eta v_k2, k1 <= k2
  for (int o = lane; o < P::n112; o += kHalf) {
    static_assert(P::K1 == P::C2, "the degree-two vech table serves the probes");
    const int eta = o % P::K2, pr = o / P::K2;
    const int k1 = rp.vp2[pr] & 0xFF, k2 = rp.vp2[pr] >> 8;
    const float acc = lds_dot<4>(s.z1c + 4 * k1, &s.qv[eta][k2][0]);
    put(P::o112 + o, -kInvSqrt5 * (k1 == k2 ? 1.0f : kSqrt2) * acc);
  }
  // (2,2,2): -sqrt(12/35) w tr(Q_a Q_b Q_c)
  if (lane < P::n222) {
    int a, b, c;
    float w;
    e222(lane, &a, &b, &c, &w);
    float tr = 0.0f;
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        float ab = 0.0f;
#pragma unroll
        for (int u = 0; u < 3; ++u) ab += s.q[a][r * 3 + u] * s.q[b][u * 3 + t];
        tr += ab * s.q[c][t * 3 + r];
      }
    put(P::o222 + lane, -kSqrt12_35 * w * tr);
  }
  if constexpr (P::L >= 3) {
    // (1,2,3) and (2,3,3): last contraction of the factored couplings
    for (int o = lane; o < P::n123 + P::n233; o += kHalf) {
      float acc = 0.0f;
      if (o < P::n123) {
        const int k1 = o / P::K2, k2 = o % P::K2;
#pragma unroll
        for (int m1 = 0; m1 < 3; ++m1) acc += s.z1[m1 * P::K1 + k1] * s.u123[m1 * P::K2 + k2];
        put(P::o123 + o, acc);
      } else {
        const int eta = o - P::n123;
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) acc += s.z2[m1 * P::K2 + eta] * s.v233[m1];
        put(P::o233 + eta, acc);
      }
    }
  }
  if constexpr (P::L >= 4) {
    // (1,3,4) [K1], (2,2,4) [k1 <= k2], (2,4,4) [K2], (3,3,4), (4,4,4)
    constexpr int n4 = P::n134 + P::n224 + P::n244 + 2;
    for (int o = lane; o < n4; o += kHalf) {
      float acc = 0.0f;
      if (o < P::n134) {
#pragma unroll
        for (int m1 = 0; m1 < 3; ++m1) acc += s.z1[m1 * P::K1 + o] * s.t134[m1];
        put(P::o134 + o, acc);
      } else if (o < P::n134 + P::n224) {
        int k1, k2;
        vech_pair(o - P::n134, P::K2, &k1, &k2);
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) {
          float r = 0.0f;
#pragma unroll
          for (int m2 = 0; m2 < 5; ++m2) r += s.t224[5 * m1 + m2] * s.z2[m2 * P::K2 + k2];
          acc += s.z2[m1 * P::K2 + k1] * r;
        }
        put(P::o224 + o - P::n134, (k1 == k2 ? 1.0f : kSqrt2) * acc);
      } else if (o < P::n134 + P::n224 + P::n244) {
        const int k1 = o - P::n134 - P::n224;
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) acc += s.z2[m1 * P::K2 + k1] * s.t244[m1];
        put(P::o244 + k1, acc);
      } else if (o == n4 - 2) {
        const DPA4C_LDS float* c = cpl + kO334;
#pragma unroll
        for (int a = 0; a < 7; ++a) {
          float r = 0.0f;
#pragma unroll
          for (int b = 0; b < 7; ++b) {
            float q = 0.0f;
#pragma unroll
            for (int e = 0; e < 9; ++e) q += c[(7 * a + b) * 9 + e] * s.xt4[e];
            r += q * s.xt3[b];
          }
          acc += r * s.xt3[a];
        }
        put(P::o334, acc);
      } else {
        const DPA4C_LDS float* c = cpl + kO444;
        for (int a = 0; a < 9; ++a) {
          float r = 0.0f;
#pragma unroll
          for (int b = 0; b < 9; ++b) {
            float q = 0.0f;
#pragma unroll
            for (int e = 0; e < 9; ++e) q += c[(9 * a + b) * 9 + e] * s.xt4[e];
            r += q * s.xt4[b];
          }
          acc += r * s.xt4[a];
        }
        put(P::o444, acc);
      }
    }
  }
  // projected quartic, Eq. (quartic), eta-major
  for (int o = lane; o < P::nPi; o += kHalf) {
    int eta = o / P::K1, k = o % P::K1;
    float acc = 0.0f;
#pragma unroll
    for (int a = 0; a < 3; ++a) acc += s.qv[eta][k][a] * s.qv[eta][k][a];
    put(P::oPi + o, acc);
  }
  wave_sync();
}

// Vector-Jacobian product of the readout: from dE/dD~ = dE/dD / sigma (LDS
// row ``d``; the producer of dE/dD applies the 1/sigma of Eq. (calibration))
// to dE/d(node state) in s.gy.  ``s`` must still hold
// what readout_forward left there for the same atom (node state and the
// forward intermediates), which are reused rather than recomputed.
template <class P>
__device__ __attribute__((noinline)) void readout_backward(DPA4C_LDS ReadoutLds<P>& s,
                                                           const DPA4C_LDS ReadoutParams<P>& rp,
                                                           DPA4C_LDS float* d) {
  const int lane = lane_of() & (kHalf - 1);
  const DPA4C_LDS float* cpl = rp.cpl;
  const float M0 = sqrtf(0.25f + s.y[0]);
  const float M1 = sqrtf(0.25f + s.y[1]);
  // --- dE/dQ_eta (3x3, not symmetrised) from (1,1,2), quartic and (2,2,2)
  if (lane < P::K2 * 9) {
    int eta = lane / 9, a = (lane % 9) / 3, b = lane % 3;
    float acc = 0.0f;
#pragma unroll
    for (int k1 = 0; k1 < P::K1; ++k1)
#pragma unroll
      for (int k2 = k1; k2 < P::K1; ++k2) {
        float jb = d[P::o112 + tri_index(k1, k2, P::K1) * P::K2 + eta];
        float f = -kInvSqrt5 * (k1 == k2 ? 1.0f : kSqrt2);
        acc += jb * f * s.z1[a * P::K1 + k1] * s.z1[b * P::K1 + k2];
      }
#pragma unroll
    for (int k = 0; k < P::K1; ++k) {
      float pb = d[P::oPi + eta * P::K1 + k];
      acc += 2.0f * pb * s.qv[eta][k][a] * s.z1[b * P::K1 + k];
    }
#pragma unroll
    for (int t = 0; t < P::n222; ++t) {
      int ia, ib, ic;
      float w;
      e222(t, &ia, &ib, &ic, &w);
      float jb = d[P::o222 + t] * (-kSqrt12_35) * w;
      // d tr(A B C) / dA = (B C)^T, / dB = (C A)^T, / dC = (A B)^T
      if (ia == eta) {
        float v = 0.0f;
#pragma unroll
        for (int u = 0; u < 3; ++u) v += s.q[ib][b * 3 + u] * s.q[ic][u * 3 + a];
        acc += jb * v;
      }
      if (ib == eta) {
        float v = 0.0f;
#pragma unroll
        for (int u = 0; u < 3; ++u) v += s.q[ic][b * 3 + u] * s.q[ia][u * 3 + a];
        acc += jb * v;
      }
      if (ic == eta) {
        float v = 0.0f;
#pragma unroll
        for (int u = 0; u < 3; ++u) v += s.q[ia][b * 3 + u] * s.q[ib][u * 3 + a];
        acc += jb * v;
      }
    }
    s.gq[eta][a * 3 + b] = acc;
  }
  // --- dE/dv (probe gradients of degree one) from (1,1,2), the quartic and (1,2,3)
  for (int o = lane; o < 3 * P::K1; o += kHalf) {
    int m = o / P::K1, k = o % P::K1;
    float acc = 0.0f;
#pragma unroll
    for (int eta = 0; eta < P::K2; ++eta) {
#pragma unroll
      for (int kp = 0; kp < P::K1; ++kp) {
        int k1 = k < kp ? k : kp, k2 = k < kp ? kp : k;
        float jb = d[P::o112 + tri_index(k1, k2, P::K1) * P::K2 + eta];
        float f = -kInvSqrt5 * (k1 == k2 ? 2.0f : kSqrt2);
        acc += jb * f * s.qv[eta][kp][m];
      }
      float pb = d[P::oPi + eta * P::K1 + k];
      float v = 0.0f;
#pragma unroll
      for (int b = 0; b < 3; ++b) v += s.q[eta][m * 3 + b] * s.qv[eta][k][b];
      acc += 2.0f * pb * v;
    }
    if constexpr (P::L >= 3) {
#pragma unroll
      for (int k2 = 0; k2 < P::K2; ++k2) acc += d[P::o123 + k * P::K2 + k2] * s.u123[m * P::K2 + k2];
    }
    if constexpr (P::L >= 4) acc += d[P::o134 + k] * s.t134[m];
    s.gz1[o] = acc;
  }
  if constexpr (P::L >= 4) {
    // adjoints of the degree-four partial contractions:
    // Tbar134[m1] = sum_k1 Jbar134[k1] Z1[m1][k1],
    // Tbar224[m1][m2] = sum_(k1<=k2) w Jbar224 Z2[m1][k1] Z2[m2][k2],
    // Tbar244[m1] = sum_k1 Jbar244[k1] Z2[m1][k1]
    for (int o = lane; o < 33; o += kHalf) {
      float acc = 0.0f;
      if (o < 3) {
#pragma unroll
        for (int k1 = 0; k1 < P::K1; ++k1) acc += d[P::o134 + k1] * s.z1[o * P::K1 + k1];
        s.tb134[o] = acc;
      } else if (o < 28) {
        const int m1 = (o - 3) / 5, m2 = (o - 3) % 5;
#pragma unroll
        for (int tt = 0; tt < P::n224; ++tt) {
          int k1, k2;
          vech_pair(tt, P::K2, &k1, &k2);
          acc += (k1 == k2 ? 1.0f : kSqrt2) * d[P::o224 + tt] * s.z2[m1 * P::K2 + k1] *
                 s.z2[m2 * P::K2 + k2];
        }
        s.tb224[o - 3] = acc;
      } else {
        const int m1 = o - 28;
#pragma unroll
        for (int k1 = 0; k1 < P::K2; ++k1) acc += d[P::o244 + k1] * s.z2[m1 * P::K2 + k1];
        s.tb244[m1] = acc;
      }
    }
  }
  if constexpr (P::L >= 3) {
    // Ubar[m1][k2] = sum_k1 Jbar123[k1][k2] Z1[m1][k1],  Vbar[m1] = sum_e Jbar233[e] Z2[m1][e]
    if (lane >= 18 && lane < 18 + 3 * P::K2) {
      const int o = lane - 18, m1 = o / P::K2, k2 = o % P::K2;
      float acc = 0.0f;
#pragma unroll
      for (int k1 = 0; k1 < P::K1; ++k1) acc += d[P::o123 + k1 * P::K2 + k2] * s.z1[m1 * P::K1 + k1];
      s.ub123[o] = acc;
    } else if (lane >= 24 && lane < 29) {
      const int m1 = lane - 24;
      float acc = 0.0f;
#pragma unroll
      for (int eta = 0; eta < P::K2; ++eta) acc += d[P::o233 + eta] * s.z2[m1 * P::K2 + eta];
      s.vb233[m1] = acc;
    }
  }
  wave_sync();
  if constexpr (P::L >= 3) {
    // Tbar[m1][m2] = sum_k2 Ubar[m1][k2] Z2[m2][k2]
    if (lane >= 16 && lane < 31) {
      const int o = lane - 16, m1 = o / 5, m2 = o % 5;
      float acc = 0.0f;
#pragma unroll
      for (int k2 = 0; k2 < P::K2; ++k2) acc += s.ub123[m1 * P::K2 + k2] * s.z2[m2 * P::K2 + k2];
      s.tb123[o] = acc;
    }
  }
  // --- dE/dz2 = E_m : dE/dQ + the generic couplings
  if (lane < 5 * P::K2) {
    int m = lane / P::K2, eta = lane % P::K2;
    float acc = stf_adjoint(s.gq[eta], m);
    if constexpr (P::L >= 3) {
#pragma unroll
      for (int m1 = 0; m1 < 3; ++m1) acc += s.ub123[m1 * P::K2 + eta] * s.t123[m1 * 5 + m];
      acc += d[P::o233 + eta] * s.v233[m];
    }
    if constexpr (P::L >= 4) {
      // (2,2,4): the pair (k1, k2) holding eta, through the symmetric T224
#pragma unroll
      for (int tt = 0; tt < P::n224; ++tt) {
        int k1, k2;
        vech_pair(tt, P::K2, &k1, &k2);
        const float jb = (k1 == k2 ? 1.0f : kSqrt2) * d[P::o224 + tt];
        if (k1 == eta) {
          float r = 0.0f;
#pragma unroll
          for (int m2 = 0; m2 < 5; ++m2) r += s.t224[5 * m + m2] * s.z2[m2 * P::K2 + k2];
          acc += jb * r;
        }
        if (k2 == eta) {
          float r = 0.0f;
#pragma unroll
          for (int m1 = 0; m1 < 5; ++m1) r += s.z2[m1 * P::K2 + k1] * s.t224[5 * m1 + m];
          acc += jb * r;
        }
      }
      acc += d[P::o244 + eta] * s.t244[m];
    }
    s.gz2[lane] = acc;
  }
  wave_sync();
  if constexpr (P::L >= 3) {
    // dE/dz3[m] = sum_{m1,m2} Tbar[m1][m2] C123[m1][m2][m] + 2 sum_m1 Vbar[m1] W[m1][m]
    if (lane < 7) {
      const int m = lane;
      float acc = 0.0f;
#pragma unroll
      for (int o = 0; o < 15; ++o) acc += s.tb123[o] * cpl[7 * o + m];
#pragma unroll
      for (int m1 = 0; m1 < 5; ++m1) acc += 2.0f * s.vb233[m1] * s.w233[m1 * 7 + m];
      if constexpr (P::L >= 4) {
        // (1,3,4): sum Tbar134[m1] C134[m1][m][e] Z4[e]; (3,3,4): 2 Jbar C334[m][b][e] Z3 Z4
#pragma unroll
        for (int m1 = 0; m1 < 3; ++m1) {
          float r = 0.0f;
#pragma unroll
          for (int e = 0; e < 9; ++e) r += cpl[kO134 + (7 * m1 + m) * 9 + e] * s.xt4[e];
          acc += s.tb134[m1] * r;
        }
        float r334 = 0.0f;
#pragma unroll
        for (int b = 0; b < 7; ++b) {
          float q = 0.0f;
#pragma unroll
          for (int e = 0; e < 9; ++e) q += cpl[kO334 + (7 * m + b) * 9 + e] * s.xt4[e];
          r334 += q * s.xt3[b];
        }
        acc += 2.0f * d[P::o334] * r334;
      }
      s.gz3[m] = acc;
    }
    if constexpr (P::L >= 4) {
      // dE/dZ4[m] from (1,3,4), (2,2,4), (2,4,4), (3,3,4), (4,4,4), then
      // dE/dX~4 = 2 Gbar4 X~4 + dE/dZ4
      if (lane >= 7 && lane < 16) {
        const int m = lane - 7;
        float acc = 0.0f;
#pragma unroll
        for (int m1 = 0; m1 < 3; ++m1) {
          float r = 0.0f;
#pragma unroll
          for (int a = 0; a < 7; ++a) r += cpl[kO134 + (7 * m1 + a) * 9 + m] * s.xt3[a];
          acc += s.tb134[m1] * r;
        }
#pragma unroll
        for (int o = 0; o < 25; ++o) acc += s.tb224[o] * cpl[kO224 + 9 * o + m];
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) {
          float r = 0.0f;
#pragma unroll
          for (int b = 0; b < 9; ++b) r += cpl[kO244 + (9 * m1 + m) * 9 + b] * s.xt4[b];
          acc += 2.0f * s.tb244[m1] * r;
        }
        float r334 = 0.0f;
#pragma unroll
        for (int a = 0; a < 7; ++a) {
          float q = 0.0f;
#pragma unroll
          for (int b = 0; b < 7; ++b) q += cpl[kO334 + (7 * a + b) * 9 + m] * s.xt3[b];
          r334 += q * s.xt3[a];
        }
        acc += d[P::o334] * r334;
        float r444 = 0.0f;
        for (int b = 0; b < 9; ++b) {
          float q = 0.0f;
#pragma unroll
          for (int e = 0; e < 9; ++e) q += cpl[kO444 + (9 * m + b) * 9 + e] * s.xt4[e];
          r444 += q * s.xt4[b];
        }
        acc += 3.0f * d[P::o444] * r444;
        s.gxt4[m] = 2.0f * d[P::oG4] * s.xt4[m] + acc;
      }
    }
    wave_sync();
  }
  // --- dE/dX~ from the Gram blocks and the probes: the Gram adjoints are
  // first expanded to full symmetric matrices (vech weights included), so
  // that each output reads two contiguous rows
  for (int o = lane; o < P::C1 * P::C1 + P::C2 * P::C2; o += kHalf) {
    if (o < P::C1 * P::C1) {
      const int c = o / P::C1, cp = o % P::C1;
      const int a = c < cp ? c : cp, b = c < cp ? cp : c;
      s.gb1[o] = d[P::oG1 + tri_index(a, b, P::C1)] * (c == cp ? 2.0f : kSqrt2);
    } else {
      const int u = o - P::C1 * P::C1, c = u / P::C2, cp = u % P::C2;
      const int a = c < cp ? c : cp, b = c < cp ? cp : c;
      s.gb2[u] = d[P::oG2 + tri_index(a, b, P::C2)] * (c == cp ? 2.0f : kSqrt2);
    }
  }
  wave_sync();
  constexpr int n1 = 3 * P::C1, n2 = 5 * P::C2, n3 = (P::L >= 3 ? 7 : 0);
  for (int o = lane; o < n1; o += kHalf) {
    const int m = o / P::C1, c = o % P::C1;
    float acc = lds_dot<P::C1>(s.gb1 + c * P::C1, s.xt1 + m * P::C1);
    if constexpr (P::kHasA1) {
      acc += lds_dot<P::K1>(s.gz1 + m * P::K1, rp.A1 + c * P::K1);
    } else {
      acc += s.gz1[m * P::K1 + c];
    }
    s.gxt1[o] = acc;
  }
  for (int o = lane; o < n2 + n3; o += kHalf) {
    if (o < n2) {
      const int m = o / P::C2, c = o % P::C2;
      float acc = lds_dot<P::C2>(s.gb2 + c * P::C2, s.xt2 + m * P::C2);
#pragma unroll
      for (int k = 0; k < P::K2; ++k) acc += s.gz2[m * P::K2 + k] * rp.A2[c * P::K2 + k];
      s.gxt2[o] = acc;
    } else {
      const int m = o - n2;
      s.gxt3[m] = 2.0f * d[P::oG3] * s.xt3[m] + s.gz3[m];
    }
  }
  wave_sync();
  // --- through the alignment (I + W) and the normalisation X = Y / M
  const float i0 = 1.0f / M0, i1 = 1.0f / M1;
  float part0 = 0.0f, part1 = 0.0f;   // sum Xbar * Y per normaliser
  for (int c = lane; c < P::C0; c += kHalf) {
    float xb = d[P::oX + c];
    s.gy[P::Y0 + c] = xb * i0;
    part0 += xb * s.y[P::Y0 + c];
  }
  constexpr int n4 = (P::L >= 4 ? 9 : 0);
  for (int o = lane; o < n1 + n2 + n3 + n4; o += kHalf) {
    float xb;
    int yi;
    if (o < n1) {
      int m = o / P::C1, c = o % P::C1;
      xb = s.gxt1[o] + lds_dot<P::C1>(s.gxt1 + m * P::C1, rp.W1 + c * P::C1);
      yi = P::Y1 + o;
    } else if (o < n1 + n2) {
      int t = o - n1, m = t / P::C2, c = t % P::C2;
      xb = s.gxt2[t] + lds_dot<P::C2>(s.gxt2 + m * P::C2, rp.W2 + c * P::C2);
      yi = P::Y2 + t;
    } else if (o < n1 + n2 + n3) {
      int m = o - n1 - n2;
      xb = s.gxt3[m];
      yi = P::Y3 + m;
    } else {
      int m = o - n1 - n2 - n3;
      xb = P::L >= 4 ? s.gxt4[m < (P::L >= 4 ? 9 : 1) ? m : 0] : 0.0f;
      yi = P::Y4 + m;
    }
    s.gy[yi] = xb * i1;
    part1 += xb * s.y[yi];
  }
  part0 = half_sum(part0);
  part1 = half_sum(part1);
  if (lane == 0) {
    float mb0 = d[P::oM0] - part0 * i0 * i0;
    float mb1 = d[P::oM1] - part1 * i1 * i1;
    s.gy[0] = mb0 * 0.5f * i0;   // M0 = sqrt(1/4 + S0)
    s.gy[1] = mb1 * 0.5f * i1;
  }
  wave_sync();
}

}  // namespace dpa4c
