// Fused backward edge kernel: readout vector-Jacobian product followed by
// the edge recomputation of Methods "Fused execution and backward
// recomputation".
//
// One wavefront per centre (four per 256-thread workgroup, never waiting for
// each other).  For centre i the wave reads the node-state gradient
// [dE/dS0, dE/dS1, dE/dY] (from the per-atom kernel), revisits the edges of
// row i, recomputes the tabulated radial maps (value and derivative), the
// pair coefficients and the envelope, and writes
//     dE/dr_ij = (dE/drho) u + (I - u u^T)(dE/du) / rho,
// with  dE/drho = sum_lmc Ybar_lmc B_lm d(chi_l psi_c)/drho
//               + Sbar0 d(chi^2)/drho + Sbar1 d(chi^4)/drho,
//       dE/du   = sum_lmc Ybar_lmc chi_l psi_c dB_lm/du.
//
// Lane k of an edge group owns the channels c = k + LPE*j.  For the
// non-scalar degrees the channel c = k contributes
//     psi_k * Q_k(u),  Q_k(u) = sum_{l>=1, m} Ybar_lmk B_lm(u),
// and Q_k is a fixed polynomial per centre: v.u (degree one), u.W u (degree
// two, W symmetric), a cubic (degree three) and a quartic (degree four).  Its
// coefficients are formed once per centre, so per edge each lane evaluates
// one short polynomial and
// its gradient instead of every harmonic.  The LPE partial sums of an edge
// are combined with a fixed DPP butterfly.
//
// The row is taken in passes of 64 edges: each lane first forms one edge's
// geometry, envelope and table row into the wave's LDS slice, so the groups
// do not repeat that work per lane; with folded tables a group requests the
// table entries of its next edge before it evaluates the current one.
//
// The gradient of an edge goes to the skin position of the edge (the force
// assembly finds a reverse gradient there with one lookup), over the
// compact records, and keeps j in the fourth component; a pass's gradients
// are stored together once its edges have run.  The passes run from the end
// of the row to its start: a skin position is never before its compact
// slot, so a gradient never lands on a record still to be read.  With VIR the
// lane that forms a gradient also adds -g_e (x) r_e (float64) to its group's
// slot in LDS; the slots are summed in group order into the atom's term W_i
// of the virial of Eq. (forces).
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "edge_math.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr int kTeam = 256;
constexpr int kWaves = kTeam / kWave;

// Four waves per SIMD for the degree-three variants without the virial
// (measured faster than three, despite a few spilled registers); the virial
// and degree-four variants would spill more and keep their natural count.
template <class P, bool VIR>
constexpr int backward_min_waves() { return P::L < 4 && !VIR ? 4 : 1; }

template <class P, bool FOLD, bool VIR>
__global__ void __launch_bounds__(kTeam, (backward_min_waves<P, VIR>())) backward_kernel(ModelDev md, int64_t n,
                                                         const int32_t* __restrict__ typ,
                                                         const int64_t* __restrict__ row_ptr,
                                                         const int32_t* __restrict__ ecount,
                                                         float4* edge,
                                                         const int32_t* __restrict__ cskin,
                                                         const float* __restrict__ node_grad,
                                                         double* __restrict__ w_atom) {
  static_assert(P::R == 0 || P::R == 4, "pair modes: 0 or 4");
  constexpr int G = kWave / P::LPE;   // edge groups in a wave
  __shared__ double wv_all[kWaves][VIR ? G : 1][9];
  // per edge of a pass: (u, 1/rho), (tau, chi, dchi, table row), (j, a_j);
  // the per-edge terms that do not depend on the lane's channel: (chi^2,
  // d chi^2/drho, the S0/S1 term, the degree-three/four part of Q_0), the
  // gradient of that part with the edge's skin position (bits), and with
  // folded tables the quintic weights (e2, e3, f2, f3)
  __shared__ float4 geo_all[kWaves][kWave];
  __shared__ float4 rad_all[kWaves][kWave];
  __shared__ int2 ids_all[kWaves][kWave];
  __shared__ float4 sc_all[kWaves][kWave];
  __shared__ float4 cb_all[kWaves][kWave];
  __shared__ float4 wt_all[kWaves][FOLD ? kWave : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int grp = lane / P::LPE;
  const int k = lane % P::LPE;
  double (*wv)[9] = wv_all[wave];
  float4* geo = geo_all[wave];
  float4* rad = rad_all[wave];
  int2* ids = ids_all[wave];
  float4* scl = sc_all[wave];
  float4* cub = cb_all[wave];
  float4* wts = wt_all[wave];
  const int T1 = md.n_types1;
  const float inv_delta = md.inv_delta;
  const int nf = md.fold_n;
  // ``typ`` holds species (clamped here) or, with folded tables, the folded
  // index of every atom
  auto type_of = [&](int64_t a) { return FOLD ? typ[a] : clamp_type(typ[a], T1); };

  for (int64_t blk = xcd_block(blockIdx.x, gridDim.x); blk * kWaves < n; blk += gridDim.x) {
    const int64_t i = blk * kWaves + wave;
    if (i >= n) break;
    const int ai = type_of(i);
    const float* gyr = node_grad + size_t(i) * P::NS;
    // per-centre coefficients in the lane's channel layout
    float gy0[P::CPL];
#pragma unroll
    for (int j = 0; j < P::CPL; ++j) gy0[j] = gyr[P::Y0 + j * P::LPE + k];
    float v1[3];
#pragma unroll
    for (int m = 0; m < 3; ++m) v1[m] = gyr[P::Y1 + m * P::C1 + k];
    float M2[6];
    {
      float w[5];
#pragma unroll
      for (int m = 0; m < 5; ++m) w[m] = k < P::C2 ? gyr[P::Y2 + m * P::C2 + k] : 0.0f;
      quad_form2(w, M2);
    }
    // channel 0's degree-three (and four) polynomial and the normaliser
    // gradients, in every lane: the per-edge pass evaluates them once per
    // edge, and only lane 0 of a group adds them
    float G3[3][6];
    {
      float w[7];
#pragma unroll
      for (int m = 0; m < 7; ++m) w[m] = P::L >= 3 ? gyr[P::Y3 + m] : 0.0f;
      cubic_form3(w, G3);
#pragma unroll
      for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int qq = 0; qq < 6; ++qq) G3[a][qq] = wave_uniform(G3[a][qq]);
    }
    float G4[P::L >= 4 ? 3 : 1][10];   // gradient of the degree-four polynomial
    if constexpr (P::L >= 4) {
      float w[9], pc[15];
#pragma unroll
      for (int m = 0; m < 9; ++m) w[m] = gyr[P::Y4 + m];
      quartic_coeffs4(w, pc);
      quartic_grad4(pc, G4);
#pragma unroll
      for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int qq = 0; qq < 10; ++qq) G4[a][qq] = wave_uniform(G4[a][qq]);
    }
    const float gs0 = wave_uniform(gyr[0]), gs1 = wave_uniform(gyr[1]);
    const float m0 = k == 0 ? 1.0f : 0.0f;

    const int64_t b = row_ptr[i];
    const int cnt = ecount[i];
    if (VIR && k == 0)
      for (int c = 0; c < 9; ++c) wv[grp][c] = 0.0;
    const float* pair_base = FOLD ? md.ftab + size_t(ai) * nf * md.n_rows * (P::C0 * kFoldWords)
                                  : md.pair + size_t(ai) * T1 * (P::C0 * P::PW);

    // Entry x of the pass (compact slot c0 + x of the row): the edge
    // gradient from its LDS entry and, with folded tables, the lane's table
    // entries ``T`` of that edge.
    auto edge_work = [&](int x, int c0, const float3* T) {
      const float4 ge = geo[x], ra = rad[x];
      const float x_ = ge.x, y = ge.y, z = ge.z, inv_rho = ge.w;
      const float tau = ra.x, chi = ra.y, dchi = ra.z;
      const bool valid = c0 + x < cnt;
      const float4 sc = scl[x];
      float a0 = 0.0f, b0 = 0.0f, psi0 = 0.0f, dpsi0 = 0.0f;
      if constexpr (FOLD) {
        // the quintic of each channel from the table of the pair (a_i, a_j)
        // (c4 and c5 below float32 resolution, not stored), power form; the
        // float16 c2, c3 enter through their scaled weights (one
        // mixed-precision FMA each).  The weighted sums a0 and b0 only
        // need the lane's coefficients contracted with dE/dY0 first,
        // A_p = sum_j Ybar0_j c_pj, and then one quintic in tau and its
        // derivative; d/drho's 1/Delta is applied once to the sums.
        const float4 wt = wts[x];
        const float e2 = wt.x, e3 = wt.y, f2 = wt.z, f3 = wt.w;
        float A[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          const float c0f = T[jj].x, c1 = T[jj].y;
          const uint32_t h23 = __float_as_uint(T[jj].z);
          const float h2 = half_lo(h23), h3 = half_hi(h23);
          if (jj == 0) {   // the amplitude of the lane's first channel itself
            psi0 = fmaf(c1, tau, c0f);
            psi0 = fmaf(h2, e2, psi0);
            psi0 = fmaf(h3, e3, psi0);
            dpsi0 = fmaf(h2, f2, c1);
            dpsi0 = fmaf(h3, f3, dpsi0);
          }
          A[0] = fmaf(gy0[jj], c0f, A[0]);
          A[1] = fmaf(gy0[jj], c1, A[1]);
          A[2] = fmaf(gy0[jj], h2, A[2]);
          A[3] = fmaf(gy0[jj], h3, A[3]);
        }
        a0 = fmaf(A[3], e3, fmaf(A[2], e2, fmaf(A[1], tau, A[0])));
        b0 = fmaf(A[3], f3, fmaf(A[2], f2, A[1])) * inv_delta;
        dpsi0 *= inv_delta;
      } else {
        const float t2 = tau * tau, t3 = t2 * tau, t4 = t2 * t2, t5 = t4 * tau;
        const float d1 = 2.0f * tau, d2 = 3.0f * t2, d3 = 4.0f * t3, d4 = 5.0f * t4;
        const int row = __float_as_int(ra.w), aj = ids[x].y;
        float q[4] = {0.f, 0.f, 0.f, 0.f}, dq[4] = {0.f, 0.f, 0.f, 0.f};
        if constexpr (P::R > 0) {
          float c[6];
          load6(md.qtab + (size_t(row) * P::R + (k < P::R ? k : 0)) * 6, c);
          const float qk = c[0] + c[1] * tau + c[2] * t2 + c[3] * t3 + c[4] * t4 + c[5] * t5;
          const float dqk = (c[1] + c[2] * d1 + c[3] * d2 + c[4] * d3 + c[5] * d4) * inv_delta;
#pragma unroll
          for (int mu = 0; mu < 4; ++mu) {
            q[mu] = __shfl(qk, mu, P::LPE);
            dq[mu] = __shfl(dqk, mu, P::LPE);
          }
        }
        const float* pc = pair_base + size_t(aj) * (P::C0 * P::PW);
        const float* gt = md.gtab + size_t(row) * (P::C0 * 6);
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          float c[6];
          load6(gt + (jj * P::LPE + k) * 6, c);
          const float gv = c[0] + c[1] * tau + c[2] * t2 + c[3] * t3 + c[4] * t4 + c[5] * t5;
          const float gd = (c[1] + c[2] * d1 + c[3] * d2 + c[4] * d3 + c[5] * d4) * inv_delta;
          const float* pp = pc + (jj * P::LPE + k) * P::PW;
          const float2 gb = *reinterpret_cast<const float2*>(pp);
          float psi = gb.x * gv + gb.y;
          float dpsi = gb.x * gd;
          if constexpr (P::R > 0) {
            const float2 u01 = *reinterpret_cast<const float2*>(pp + 2);
            const float2 u23 = *reinterpret_cast<const float2*>(pp + 4);
            psi += u01.x * q[0] + u01.y * q[1] + u23.x * q[2] + u23.y * q[3];
            dpsi += u01.x * dq[0] + u01.y * dq[1] + u23.x * dq[2] + u23.y * dq[3];
          }
          a0 += gy0[jj] * psi;
          b0 += gy0[jj] * dpsi;
          if (jj == 0) {
            psi0 = psi;
            dpsi0 = dpsi;
          }
        }
      }
      // Q_k(u) and its gradient: the lane's degree-one and degree-two parts
      // here, channel 0's degree-three (and four) part from the pass
      float gq[3];
      gq[0] = M2[0] * x_ + M2[3] * y + M2[5] * z;
      gq[1] = M2[3] * x_ + M2[1] * y + M2[4] * z;
      gq[2] = M2[5] * x_ + M2[4] * y + M2[2] * z;
      const float4 cb = cub[x];
      // Q = v.u + (1/2) u.M u + (1/3) u.grad P3 + (1/4) u.grad P4 (Euler's
      // relation per degree)
      const float Q = (v1[0] * x_ + v1[1] * y + v1[2] * z) +
                      0.5f * (gq[0] * x_ + gq[1] * y + gq[2] * z) + m0 * sc.w;
      const float chi2 = sc.x, dchi2 = sc.y;
      float drho = dchi * a0 + chi * b0 + Q * (dchi2 * psi0 + chi2 * dpsi0) + m0 * sc.z;
      const float wu = chi2 * psi0;
      float dux = wu * (v1[0] + gq[0] + m0 * cb.x);
      float duy = wu * (v1[1] + gq[1] + m0 * cb.y);
      float duz = wu * (v1[2] + gq[2] + m0 * cb.z);
      if (!valid) drho = dux = duy = duz = 0.0f;
      drho = group_sum<P::LPE>(drho);
      dux = group_sum<P::LPE>(dux);
      duy = group_sum<P::LPE>(duy);
      duz = group_sum<P::LPE>(duz);
      if (valid && k == 0) {
        const float udu = x_ * dux + y * duy + z * duz;
        const float gx = drho * x_ + (dux - udu * x_) * inv_rho;
        const float gy_ = drho * y + (duy - udu * y) * inv_rho;
        const float gz = drho * z + (duz - udu * z) * inv_rho;
        // to the entry's LDS slot (its geometry is no longer needed): the
        // pass's gradients are stored together once every edge has run
        geo[x] = make_float4(gx, gy_, gz, __int_as_float(ids[x].x));
        if (VIR) {   // LDS adds to the group's own slot: one writer, program order
          const float rho = __builtin_amdgcn_rcpf(inv_rho);   // hardware reciprocal, 1 ulp
          const float ga[3] = {gx, gy_, gz};
          const float rb[3] = {x_ * rho, y * rho, z * rho};
#pragma unroll
          for (int a = 0; a < 3; ++a)
#pragma unroll
            for (int c = 0; c < 3; ++c) atomicAdd(&wv[grp][3 * a + c], -(double(ga[a]) * double(rb[c])));
        }
      }
    };
    // the lane's folded table entries of entry x of the pass
    auto load_rows = [&](int x, float3* T) {
      load_fold_row<P::LPE, P::CPL>(
          pair_base + size_t(__float_as_int(rad[x].w)) * (P::C0 * kFoldWords), k, T);
    };

    // The row in passes of 64 edges: each lane first reads one record and
    // forms its edge's geometry, envelope and table row into the wave's LDS
    // slice (entries past the row get chi = 0 and table row 0), then the
    // groups take the pass's edges.
    for (int c0 = ((cnt - 1) / kWave) * kWave; cnt > 0 && c0 >= 0; c0 -= kWave) {
      const int np = cnt - c0 < kWave ? cnt - c0 : kWave;
      {
        float4 ge = make_float4(0.f, 0.f, 0.f, 1.0f), ra = make_float4(0.f, 0.f, 0.f, 0.f);
        float4 sc = make_float4(0.f, 0.f, 0.f, 0.f), cb = sc, wt = sc;
        int2 id = make_int2(0, 0);
        int sk = 0;
        if (lane < np) {
          const float4 rec = edge[b + c0 + lane];
          sk = cskin[b + c0 + lane];
          const EdgeGeom g = edge_geom(rec.x, rec.y, rec.z);
          float chi, dchi, tau;
          envelope(g.rho, md.inv_rc, &chi, &dchi);
          const int row = table_row(g.rho, inv_delta, md.n_rows, &tau);
          const int j = __float_as_int(rec.w);
          const int aj = type_of(j);
          ge = make_float4(g.ux, g.uy, g.uz, g.inv_rho);
          ra = make_float4(tau, chi, dchi, __int_as_float(FOLD ? aj * md.n_rows + row : row));
          id = make_int2(j, aj);
          const float x_ = g.ux, y = g.uy, z = g.uz;
          const float chi2 = chi * chi, dchi2 = 2.0f * chi * dchi;
          float c3[3] = {0.f, 0.f, 0.f};
          if constexpr (P::L >= 3) {
            const float mono[6] = {x_ * x_, x_ * y, x_ * z, y * y, y * z, z * z};
#pragma unroll
            for (int a = 0; a < 3; ++a) {
#pragma unroll
              for (int qq = 0; qq < 6; ++qq) c3[a] += G3[a][qq] * mono[qq];
            }
          }
          float c4[3] = {0.f, 0.f, 0.f};   // grad P4
          if constexpr (P::L >= 4) {
            float mono3[10];
            cubic_monomials(x_, y, z, mono3);
#pragma unroll
            for (int a = 0; a < 3; ++a) {
#pragma unroll
              for (int qq = 0; qq < 10; ++qq) c4[a] += G4[a][qq] * mono3[qq];
            }
          }
          float q0 = (1.0f / 3.0f) * (c3[0] * x_ + c3[1] * y + c3[2] * z);
          if constexpr (P::L >= 4) q0 += 0.25f * (c4[0] * x_ + c4[1] * y + c4[2] * z);
          sc = make_float4(chi2, dchi2, gs0 * dchi2 + gs1 * 2.0f * chi2 * dchi2, q0);
          cb = make_float4(c3[0] + c4[0], c3[1] + c4[1], c3[2] + c4[2], __int_as_float(sk));
          if constexpr (FOLD) {
            const float t2 = tau * tau, t3 = t2 * tau;
            wt = make_float4(md.c_inv[0] * t2, md.c_inv[1] * t3, md.c_inv[0] * (2.0f * tau),
                             md.c_inv[1] * (3.0f * t2));
          }
        }
        geo[lane] = ge;
        rad[lane] = ra;
        ids[lane] = id;
        scl[lane] = sc;
        cub[lane] = cb;
        if constexpr (FOLD) wts[lane] = wt;
      }
      wave_sync();
      if constexpr (FOLD) {
        // the table entries of a group's next edge are requested before its
        // current edge is evaluated (two register sets, used in turn)
        float3 TA[P::CPL], TB[P::CPL];
        load_rows(grp, TA);
        for (int base = 0; base < np; base += 2 * G) {
          if (base + G < np) load_rows(base + G + grp, TB);
          edge_work(base + grp, c0, TA);
          if (base + G >= np) break;
          if (base + 2 * G < np) load_rows(base + 2 * G + grp, TA);
          edge_work(base + G + grp, c0, TB);
        }
      } else {
        for (int base = 0; base < np; base += G) edge_work(base + grp, c0, nullptr);
      }
      wave_sync();
      // every record of the pass was read before its edges ran
      if (lane < np) edge[b + __float_as_int(cub[lane].w)] = geo[lane];
      wave_sync();   // the LDS entries are rewritten by the next pass
    }
    if (VIR) {
      wave_sync();
      if (lane < 9) {
        double s = 0.0;
        for (int q = 0; q < G; ++q) s += wv[q][lane];
        w_atom[9 * i + lane] = s;
      }
      wave_sync();   // the slots are cleared for the next row
    }
  }
}

template <class P>
int launch(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
           const int64_t* row_ptr, const int32_t* ecount, float4* edge, const int32_t* cskin,
           const float* node_grad, double* w_atom, hipStream_t st) {
  int64_t blocks = (n + kWaves - 1) / kWaves;   // a wave per centre
  blocks = blocks < 65536 ? blocks : 65536;
  if (blocks < 1) return 0;
  const int32_t* typ = fidx ? fidx : species;
  const dim3 grid(static_cast<unsigned>(blocks)), block(kTeam);
  if (fidx && w_atom)
    hipLaunchKernelGGL((backward_kernel<P, true, true>), grid, block, 0, st, m->dev(), n, typ,
                       row_ptr, ecount, edge, cskin, node_grad, w_atom);
  else if (fidx)
    hipLaunchKernelGGL((backward_kernel<P, true, false>), grid, block, 0, st, m->dev(), n, typ,
                       row_ptr, ecount, edge, cskin, node_grad, w_atom);
  else if (w_atom)
    hipLaunchKernelGGL((backward_kernel<P, false, true>), grid, block, 0, st, m->dev(), n, typ,
                       row_ptr, ecount, edge, cskin, node_grad, w_atom);
  else
    hipLaunchKernelGGL((backward_kernel<P, false, false>), grid, block, 0, st, m->dev(), n, typ,
                       row_ptr, ecount, edge, cskin, node_grad, w_atom);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_backward(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
                    const int64_t* row_ptr, const int32_t* ecount, float4* edge,
                    const int32_t* cskin, const float* node_grad, double* w_atom, hipStream_t st) {
  const int rc = with_profile(m->C0, m->L, m->R, m->F, [&](auto p, auto) {
    return launch<decltype(p)>(m, n, species, fidx, row_ptr, ecount, edge, cskin, node_grad,
                               w_atom, st);
  });
  if (rc == kNoProfile) {
    set_error("backward: profile not compiled");
    return DPA4C_ERR_UNSUPPORTED;
  }
  return rc;
}

}  // namespace dpa4c
