// Fused forward edge kernel: featurisation, single aggregation and readout.
//
// Methods Eqs. (edge-geometry) .. (moments): for every centre i, the edges of
// its row are scanned once; per edge the envelope, the tabulated radial maps
// g and q, the cached pair coefficients gamma, beta, U, the amplitude psi and
// the harmonics are formed in registers and accumulated into the node state
// [sum chi^2, sum chi^4, Y_lmc].  No per-edge quantity is written to memory.
// The readout (Eqs. (alignment) .. (calibration)) then runs on the same
// wavefront and writes the calibrated descriptor D_i.
//
// Mapping: one wavefront per centre.  The 64 lanes form EPW groups of
// LPE = C1 lanes; each group takes one edge at a time and lane k of a group
// owns the channels c = k + LPE*j.  Groups are combined at the end of the
// row with a fixed xor butterfly, so the node state is the same bits on
// every run.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "edge_math.h"
#include "launch.h"
#include "readout.h"

namespace dpa4c {

namespace {

constexpr int kBlock = 256;
constexpr int kWpb = kBlock / kWave;

template <class P>
__global__ void __launch_bounds__(kBlock) forward_kernel(ModelDev md, int64_t n,
                                                         const int32_t* __restrict__ species,
                                                         const int64_t* __restrict__ row_ptr,
                                                         const int32_t* __restrict__ ecount,
                                                         const float4* __restrict__ edge,
                                                         float* __restrict__ node,
                                                         float* __restrict__ desc) {
  __shared__ ReadoutLds<P> lds_all[kWpb];
  ReadoutLds<P>& s = lds_all[threadIdx.x / kWave];
  const int lane = lane_of();
  const int grp = lane / P::LPE;
  const int k = lane % P::LPE;
  const int64_t nwaves = int64_t(gridDim.x) * kWpb;
  const int T1 = md.n_types1;
  const float inv_delta = md.inv_delta;

  for (int64_t i = blockIdx.x * int64_t(kWpb) + threadIdx.x / kWave; i < n; i += nwaves) {
    const int ai = clamp_type(species[i], T1);
    const int64_t b = row_ptr[i];
    const int cnt = ecount[i];
    float acc0[P::CPL];
#pragma unroll
    for (int j = 0; j < P::CPL; ++j) acc0[j] = 0.0f;
    float acc1[3] = {0.f, 0.f, 0.f};
    float acc2[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
    float acc3[7] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float s0 = 0.0f, s1 = 0.0f;
    const float* pair_base = md.pair + size_t(ai) * T1 * (P::C0 * P::PW);

    for (int base = 0; base < cnt; base += P::EPW) {
      const int el = base + grp;
      if (el < cnt) {
        const float4 rec = edge[b + el];
        const int j = __float_as_int(rec.w);
        const int aj = clamp_type(species[j], T1);
        const EdgeGeom g = edge_geom(rec.x, rec.y, rec.z);
        float chi;
        envelope(g.rho, md.r_c, &chi, nullptr);
        float tau;
        const int row = table_row(g.rho, inv_delta, md.n_rows, &tau);
        float q[P::R > 0 ? P::R : 1];
        if constexpr (P::R > 0) {
#pragma unroll
          for (int mu = 0; mu < P::R; ++mu) {
            float c[6];
            load6(md.qtab + (size_t(row) * P::R + mu) * 6, c);
            q[mu] = quintic_val(c, tau);
          }
        }
        const float* pc = pair_base + size_t(aj) * (P::C0 * P::PW);
        const float* gt = md.gtab + size_t(row) * (P::C0 * 6);
        float psi0 = 0.0f;
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          float c[6];
          load6(gt + (jj * P::LPE + k) * 6, c);
          const float gv = quintic_val(c, tau);
          const float* pp = pc + (jj * P::LPE + k) * P::PW;
          float psi = pp[0] * gv + pp[1];
          if constexpr (P::R > 0) {
#pragma unroll
            for (int mu = 0; mu < P::R; ++mu) psi += pp[2 + mu] * q[mu];
          }
          acc0[jj] += chi * psi;
          if (jj == 0) psi0 = psi;
        }
        const float chi2 = chi * chi;
        s0 += chi2;
        s1 += chi2 * chi2;
        const float w = chi2 * psi0;
        acc1[0] += w * g.ux;
        acc1[1] += w * g.uy;
        acc1[2] += w * g.uz;
        if (k < P::C2) {
          float b2[5];
          harm2(g.ux, g.uy, g.uz, b2);
#pragma unroll
          for (int m = 0; m < 5; ++m) acc2[m] += w * b2[m];
        }
        if constexpr (P::L >= 3) {
          if (k == 0) {
            float b3[7];
            harm3(g.ux, g.uy, g.uz, b3);
#pragma unroll
            for (int m = 0; m < 7; ++m) acc3[m] += w * b3[m];
          }
        }
      }
    }
    // combine the edge groups (fixed butterfly)
#pragma unroll
    for (int off = P::LPE; off < kWave; off <<= 1) {
#pragma unroll
      for (int j = 0; j < P::CPL; ++j) acc0[j] += __shfl_xor(acc0[j], off);
#pragma unroll
      for (int m = 0; m < 3; ++m) acc1[m] += __shfl_xor(acc1[m], off);
#pragma unroll
      for (int m = 0; m < 5; ++m) acc2[m] += __shfl_xor(acc2[m], off);
      if constexpr (P::L >= 3) {
#pragma unroll
        for (int m = 0; m < 7; ++m) acc3[m] += __shfl_xor(acc3[m], off);
      }
      s0 += __shfl_xor(s0, off);
      s1 += __shfl_xor(s1, off);
    }
    if (grp == 0) {
#pragma unroll
      for (int j = 0; j < P::CPL; ++j) s.y[P::Y0 + j * P::LPE + k] = acc0[j];
#pragma unroll
      for (int m = 0; m < 3; ++m) s.y[P::Y1 + m * P::C1 + k] = acc1[m];
      if (k < P::C2) {
#pragma unroll
        for (int m = 0; m < 5; ++m) s.y[P::Y2 + m * P::C2 + k] = acc2[m];
      }
      if constexpr (P::L >= 3) {
        if (k == 0) {
#pragma unroll
          for (int m = 0; m < 7; ++m) s.y[P::Y3 + m] = acc3[m];
        }
      }
      if (k == 0) {
        s.y[0] = s0;
        s.y[1] = s1;
      }
    }
    wave_sync();
    float* nrow = node + size_t(i) * P::NS;
    for (int t = lane; t < P::NS; t += kWave) nrow[t] = s.y[t];
    readout_forward<P>(s, md, ai, desc + size_t(i) * P::DSTR);
  }
}

template <class P>
int launch(const dpa4c_model* m, int64_t n, const int32_t* species, const int64_t* row_ptr,
           const int32_t* ecount, const float4* edge, float* node, float* desc, hipStream_t st) {
  int64_t blocks = (n + kWpb - 1) / kWpb;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(forward_kernel<P>, dim3(blocks), dim3(kBlock), 0, st, m->dev(), n, species,
                     row_ptr, ecount, edge, node, desc);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_forward(const dpa4c_model* m, int64_t n, const int32_t* species,
                   const int64_t* row_ptr, const int32_t* ecount, const float4* edge,
                   float* node, float* desc, hipStream_t st) {
  if (m->C0 == 32) return launch<SmallProfile>(m, n, species, row_ptr, ecount, edge, node, desc, st);
  return launch<FullProfile>(m, n, species, row_ptr, ecount, edge, node, desc, st);
}

}  // namespace dpa4c
