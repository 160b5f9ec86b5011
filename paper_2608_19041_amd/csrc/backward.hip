// Fused backward edge kernel: readout vector-Jacobian product followed by
// the edge recomputation of Methods "Fused execution and backward
// recomputation".
//
// For centre i the kernel first turns dE/dD_i into the node-state gradient
// [dE/dS0, dE/dS1, dE/dY] (readout VJP), then revisits the edges of row i,
// recomputes the tabulated radial maps (value and derivative), the pair
// coefficients, the envelope and the harmonics, and writes
//     dE/dr_ij = (dE/drho) u + (I - u u^T)(dE/du) / rho,
// with  dE/drho = sum_lmc Ybar_lmc B_lm d(chi_l psi_c)/drho
//               + Sbar0 d(chi^2)/drho + Sbar1 d(chi^4)/drho,
//       dE/du   = sum_lmc Ybar_lmc chi_l psi_c dB_lm/du.
// Each lane forms its partial sums over the channels it owns; the LPE lanes
// of an edge group combine them with a fixed xor butterfly.
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
__global__ void __launch_bounds__(kBlock) backward_kernel(ModelDev md, int64_t n,
                                                          const int32_t* __restrict__ species,
                                                          const int64_t* __restrict__ row_ptr,
                                                          const int32_t* __restrict__ ecount,
                                                          const float4* __restrict__ edge,
                                                          const float* __restrict__ node,
                                                          const float* __restrict__ dD,
                                                          float4* __restrict__ grad) {
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
    const float* nrow = node + size_t(i) * P::NS;
    for (int t = lane; t < P::NS; t += kWave) s.y[t] = nrow[t];
    wave_sync();
    readout_backward<P>(s, md, dD + size_t(i) * P::DSTR);
    // node-state gradient into registers, in the lane's channel layout
    float gy0[P::CPL];
#pragma unroll
    for (int j = 0; j < P::CPL; ++j) gy0[j] = s.gy[P::Y0 + j * P::LPE + k];
    float gy1[3], gy2[5], gy3[7];
#pragma unroll
    for (int m = 0; m < 3; ++m) gy1[m] = s.gy[P::Y1 + m * P::C1 + k];
#pragma unroll
    for (int m = 0; m < 5; ++m) gy2[m] = k < P::C2 ? s.gy[P::Y2 + m * P::C2 + k] : 0.0f;
#pragma unroll
    for (int m = 0; m < 7; ++m) gy3[m] = (P::L >= 3 && k == 0) ? s.gy[P::Y3 + m] : 0.0f;
    const float gs0 = s.gy[0], gs1 = s.gy[1];
    wave_sync();

    const int64_t b = row_ptr[i];
    const int cnt = ecount[i];
    const float* pair_base = md.pair + size_t(ai) * T1 * (P::C0 * P::PW);
    for (int base = 0; base < cnt; base += P::EPW) {
      const int el = base + grp;
      const bool valid = el < cnt;
      float drho = 0.0f, dux = 0.0f, duy = 0.0f, duz = 0.0f;
      EdgeGeom g{1.0f, 0.0f, 0.0f, 1.0f, 1.0f};
      if (valid) {
        const float4 rec = edge[b + el];
        const int j = __float_as_int(rec.w);
        const int aj = clamp_type(species[j], T1);
        g = edge_geom(rec.x, rec.y, rec.z);
        float chi, dchi;
        envelope(g.rho, md.r_c, &chi, &dchi);
        float tau;
        const int row = table_row(g.rho, inv_delta, md.n_rows, &tau);
        float q[P::R > 0 ? P::R : 1], dq[P::R > 0 ? P::R : 1];
        if constexpr (P::R > 0) {
#pragma unroll
          for (int mu = 0; mu < P::R; ++mu) {
            float c[6], v, d;
            load6(md.qtab + (size_t(row) * P::R + mu) * 6, c);
            quintic_val_der(c, tau, &v, &d);
            q[mu] = v;
            dq[mu] = d * inv_delta;
          }
        }
        const float* pc = pair_base + size_t(aj) * (P::C0 * P::PW);
        const float* gt = md.gtab + size_t(row) * (P::C0 * 6);
        float a0 = 0.0f, b0 = 0.0f, psi0 = 0.0f, dpsi0 = 0.0f;
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          float c[6], gv, gd;
          load6(gt + (jj * P::LPE + k) * 6, c);
          quintic_val_der(c, tau, &gv, &gd);
          gd *= inv_delta;
          const float* pp = pc + (jj * P::LPE + k) * P::PW;
          float psi = pp[0] * gv + pp[1];
          float dpsi = pp[0] * gd;
          if constexpr (P::R > 0) {
#pragma unroll
            for (int mu = 0; mu < P::R; ++mu) {
              psi += pp[2 + mu] * q[mu];
              dpsi += pp[2 + mu] * dq[mu];
            }
          }
          a0 += gy0[jj] * psi;
          b0 += gy0[jj] * dpsi;
          if (jj == 0) {
            psi0 = psi;
            dpsi0 = dpsi;
          }
        }
        // degree 0: weight chi
        drho = dchi * a0 + chi * b0;
        // degrees >= 1: weight chi^2, channel c = k
        const float chi2 = chi * chi, dchi2 = 2.0f * chi * dchi;
        {
          const float u[3] = {g.ux, g.uy, g.uz};
#pragma unroll
          for (int m = 0; m < 3; ++m) {
            const float a = gy1[m] * psi0, bb = gy1[m] * dpsi0;
            drho += u[m] * (dchi2 * a + chi2 * bb);
          }
          dux += chi2 * gy1[0] * psi0;
          duy += chi2 * gy1[1] * psi0;
          duz += chi2 * gy1[2] * psi0;
        }
        if (k < P::C2) {
          float b2[5], g2[5][3];
          harm2(g.ux, g.uy, g.uz, b2);
          harm2_grad(g.ux, g.uy, g.uz, g2);
#pragma unroll
          for (int m = 0; m < 5; ++m) {
            const float a = gy2[m] * psi0, bb = gy2[m] * dpsi0;
            drho += b2[m] * (dchi2 * a + chi2 * bb);
            dux += chi2 * a * g2[m][0];
            duy += chi2 * a * g2[m][1];
            duz += chi2 * a * g2[m][2];
          }
        }
        if constexpr (P::L >= 3) {
          if (k == 0) {
            float b3[7], g3[7][3];
            harm3(g.ux, g.uy, g.uz, b3);
            harm3_grad(g.ux, g.uy, g.uz, g3);
#pragma unroll
            for (int m = 0; m < 7; ++m) {
              const float a = gy3[m] * psi0, bb = gy3[m] * dpsi0;
              drho += b3[m] * (dchi2 * a + chi2 * bb);
              dux += chi2 * a * g3[m][0];
              duy += chi2 * a * g3[m][1];
              duz += chi2 * a * g3[m][2];
            }
          }
        }
        if (k == 0) drho += gs0 * dchi2 + gs1 * 2.0f * chi2 * dchi2;   // d(chi^4) = 2 chi^2 d(chi^2)
      }
      // combine the lanes of the edge group (fixed butterfly)
#pragma unroll
      for (int off = 1; off < P::LPE; off <<= 1) {
        drho += __shfl_xor(drho, off);
        dux += __shfl_xor(dux, off);
        duy += __shfl_xor(duy, off);
        duz += __shfl_xor(duz, off);
      }
      if (valid && k == 0) {
        const float udu = g.ux * dux + g.uy * duy + g.uz * duz;
        const float gx = drho * g.ux + (dux - udu * g.ux) * g.inv_rho;
        const float gyv = drho * g.uy + (duy - udu * g.uy) * g.inv_rho;
        const float gz = drho * g.uz + (duz - udu * g.uz) * g.inv_rho;
        grad[b + el] = make_float4(gx, gyv, gz, 0.0f);
      }
    }
  }
}

template <class P>
int launch(const dpa4c_model* m, int64_t n, const int32_t* species, const int64_t* row_ptr,
           const int32_t* ecount, const float4* edge, const float* node, const float* dD,
           float4* grad, hipStream_t st) {
  int64_t blocks = (n + kWpb - 1) / kWpb;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(backward_kernel<P>, dim3(blocks), dim3(kBlock), 0, st, m->dev(), n, species,
                     row_ptr, ecount, edge, node, dD, grad);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_backward(const dpa4c_model* m, int64_t n, const int32_t* species,
                    const int64_t* row_ptr, const int32_t* ecount, const float4* edge,
                    const float* node, const float* dD, float4* grad, hipStream_t st) {
  if (m->C0 == 32)
    return launch<SmallProfile>(m, n, species, row_ptr, ecount, edge, node, dD, grad, st);
  return launch<FullProfile>(m, n, species, row_ptr, ecount, edge, node, dD, grad, st);
}

}  // namespace dpa4c
