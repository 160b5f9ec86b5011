// Fused forward edge kernel: compaction, featurisation and single
// aggregation.
//
// Methods Eqs. (edge-geometry) .. (moments): for every centre i, the skin
// row is first compacted to the edges inside r_c (compact.h), then those
// edges are scanned once; per edge the envelope, the tabulated radial maps
// g and q, the cached pair coefficients gamma, beta, U, the amplitude psi and
// the harmonics are formed in registers and accumulated into the node state
// [sum chi^2, sum chi^4, Y_lmc].  Apart from the compacted edge records, no
// per-edge quantity is written to memory.
// The readout runs in the per-atom kernel.
//
// Mapping: one 256-thread workgroup per centre (striding over centres).  The
// threads form groups of LPE = C1 lanes; each group takes one edge at a time
// and lane k of a group owns the channels c = k + LPE*j, so every channel
// c < C1 of the non-scalar degrees sits in slot j = 0.  Groups are combined
// at the end of the row in a fixed order (xor butterfly inside a wave, then
// the four waves in order), so the node state is the same bits on every run.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "compact.h"
#include "edge_math.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr int kTeam = 256;
constexpr int kWaves = kTeam / kWave;

template <class P, bool FOLD>
__global__ void __launch_bounds__(kTeam) forward_kernel(ModelDev md, int64_t n,
                                                        const int32_t* __restrict__ typ,
                                                        const int64_t* __restrict__ row_ptr,
                                                        CompactArgs ca,
                                                        float* __restrict__ node) {
  constexpr int G = kTeam / P::LPE;          // edge groups in the workgroup
  __shared__ float part[kWaves][P::NS];
  __shared__ int wtot[kWaves];
  const float4* __restrict__ edge = ca.edge;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int grp = tid / P::LPE;
  const int k = tid % P::LPE;
  const int T1 = md.n_types1;
  const float inv_delta = md.inv_delta;
  const int nf = md.fold_n;
  // ``typ`` holds species (clamped here) or, with folded tables, the folded
  // index of every atom
  auto type_of = [&](int64_t a) { return FOLD ? typ[a] : clamp_type(typ[a], T1); };

  for (int64_t i = xcd_block(blockIdx.x, gridDim.x); i < n; i += gridDim.x) {
    const int ai = type_of(i);
    const int64_t b = row_ptr[i];
    // the row's edges inside r_c, compacted to the head of its skin row
    const int cnt = compact_row<kTeam>(ca, n, i, b, row_ptr[i + 1], wtot);
    float acc0[P::CPL];
#pragma unroll
    for (int j = 0; j < P::CPL; ++j) acc0[j] = 0.0f;
    float acc1[3] = {0.f, 0.f, 0.f};
    float acc2[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
    float acc3[7] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float acc4[P::L >= 4 ? 9 : 1];
#pragma unroll
    for (int m = 0; m < (P::L >= 4 ? 9 : 1); ++m) acc4[m] = 0.0f;
    float s0 = 0.0f, s1 = 0.0f;
    const float* pair_base = FOLD ? md.ftab + size_t(ai) * nf * md.n_rows * (P::C0 * kFoldWords)
                                  : md.pair + size_t(ai) * T1 * (P::C0 * P::PW);
    const float w2mask = k < P::C2 ? 1.0f : 0.0f;
    const float w3mask = k == 0 ? 1.0f : 0.0f;

    // Two-stage software pipeline over the rounds of G edges: the record of
    // round r+2 and the neighbour species of round r+1 are requested while
    // round r computes, so a round waits only for its table and pair rows.
    // Records are read only inside [0, cnt) of the row.
    // The lanes of a group share one edge, so only its lane 0 reads the
    // record and the neighbour type; they reach the other lanes by a group
    // broadcast when the round uses them (rec_nn and aj_n hold lane 0's
    // values until then).
    const float4* erow = edge + b;
    const bool lead = k == 0;
    float4 rec_n = make_float4(0.f, 0.f, 0.f, 0.f), rec_nn = rec_n;
    int aj_n = ai;
    if (cnt > 0) {
      if (lead) rec_n = erow[grp < cnt ? grp : 0];
      rec_n = group_bcast<P::LPE>(rec_n);
      aj_n = (lead && grp < cnt) ? type_of(__float_as_int(rec_n.w)) : ai;
      if (lead && G < cnt) rec_nn = erow[grp + G < cnt ? grp + G : 0];
    }
    for (int base = 0; base < cnt; base += G) {
      const int el = base + grp;
      const bool valid = el < cnt;
      const float4 rec = rec_n;
      const int aj = __shfl(aj_n, 0, P::LPE);
      if (base + G < cnt) {
        const int el1 = el + G, el2 = el + 2 * G;
        rec_n = group_bcast<P::LPE>(rec_nn);
        aj_n = (lead && el1 < cnt) ? type_of(__float_as_int(rec_n.w)) : ai;
        if (lead && base + 2 * G < cnt) rec_nn = erow[el2 < cnt ? el2 : 0];
      }
      const EdgeGeom g = edge_geom(rec.x, rec.y, rec.z);
      float chi;
      envelope(g.rho, md.inv_rc, &chi, nullptr);
      if (!valid) chi = 0.0f;
      float tau;
      const int row = table_row(g.rho, inv_delta, md.n_rows, &tau);
      float psi0 = 0.0f;
      if constexpr (FOLD) {
        // one quintic per channel from the table of the pair (a_i, a_j)
        // power form with the float16 c2 .. c5 scaled through their weights
        // e_n = tau^n / s_n (one mixed-precision FMA each)
        const float* ft = pair_base + (size_t(aj) * md.n_rows + row) * (P::C0 * kFoldWords);
        const float t2 = tau * tau, t3 = t2 * tau;
        const float e2 = md.c_inv[0] * t2, e3 = md.c_inv[1] * t3;
        const float e4 = md.c_inv[2] * (t2 * t2), e5 = md.c_inv[3] * (t2 * t3);
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          float c0, c1;
          uint32_t h23, h45;
          load_folded(ft + jj * P::LPE * kFoldWords, k, &c0, &c1, &h23, &h45);
          float psi = fmaf(c1, tau, c0);
          psi = fmaf(half_lo(h23), e2, psi);
          psi = fmaf(half_hi(h23), e3, psi);
          psi = fmaf(half_lo(h45), e4, psi);
          psi = fmaf(half_hi(h45), e5, psi);
          acc0[jj] += chi * psi;
          if (jj == 0) psi0 = psi;
        }
      } else {
        float q[P::R > 0 ? P::R : 1];
        if constexpr (P::R > 0) {
          // lane k < R evaluates q_k; the group shares it
          float c[6];
          load6(md.qtab + (size_t(row) * P::R + (k < P::R ? k : 0)) * 6, c);
          const float qk = quintic_val(c, tau);
#pragma unroll
          for (int mu = 0; mu < P::R; ++mu) q[mu] = __shfl(qk, mu, P::LPE);
        }
        const float* pc = pair_base + size_t(aj) * (P::C0 * P::PW);
        const float* gt = md.gtab + size_t(row) * (P::C0 * 6);
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          float c[6];
          load6(gt + (jj * P::LPE + k) * 6, c);
          const float gv = quintic_val(c, tau);
          const float* pp = pc + (jj * P::LPE + k) * P::PW;
          const float2 gb = *reinterpret_cast<const float2*>(pp);
          float psi = gb.x * gv + gb.y;
          if constexpr (P::R > 0) {
            const float2 u01 = *reinterpret_cast<const float2*>(pp + 2);
            const float2 u23 = *reinterpret_cast<const float2*>(pp + 4);
            psi += u01.x * q[0] + u01.y * q[1] + u23.x * q[2] + u23.y * q[3];
          }
          acc0[jj] += chi * psi;
          if (jj == 0) psi0 = psi;
        }
      }
      const float chi2 = chi * chi;
      s0 += chi2;
      s1 += chi2 * chi2;
      const float w = chi2 * psi0;
      acc1[0] += w * g.ux;
      acc1[1] += w * g.uy;
      acc1[2] += w * g.uz;
      float b2[5];
      harm2_h(g.ux, g.uy, g.uz, b2);
      const float w2 = w * w2mask;
#pragma unroll
      for (int m = 0; m < 5; ++m) acc2[m] += w2 * b2[m];
      if constexpr (P::L >= 3) {
        float b3[7];
        harm3_h(g.ux, g.uy, g.uz, b3);
        const float w3 = w * w3mask;
#pragma unroll
        for (int m = 0; m < 7; ++m) acc3[m] += w3 * b3[m];
      }
      if constexpr (P::L >= 4) {   // degree four: one channel, as degree three
        float b4[9];
        harm4_h(g.ux, g.uy, g.uz, b4);
        const float w4 = w * w3mask;
#pragma unroll
        for (int m = 0; m < 9; ++m) acc4[m] += w4 * b4[m];
      }
    }
    // combine the groups of a wave (fixed xor butterfly over the group index)
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
      if constexpr (P::L >= 4) {
#pragma unroll
        for (int m = 0; m < 9; ++m) acc4[m] += __shfl_xor(acc4[m], off);
      }
      s0 += __shfl_xor(s0, off);
      s1 += __shfl_xor(s1, off);
    }
    if (lane < P::LPE) {
      float* pw = part[wave];
#pragma unroll
      for (int j = 0; j < P::CPL; ++j) pw[P::Y0 + j * P::LPE + k] = acc0[j];
#pragma unroll
      for (int m = 0; m < 3; ++m) pw[P::Y1 + m * P::C1 + k] = acc1[m];
      if (k < P::C2) {
#pragma unroll
        for (int m = 0; m < 5; ++m) pw[P::Y2 + m * P::C2 + k] = acc2[m];
      }
      if constexpr (P::L >= 3) {
        if (k == 0) {
#pragma unroll
          for (int m = 0; m < 7; ++m) pw[P::Y3 + m] = acc3[m];
        }
      }
      if constexpr (P::L >= 4) {
        if (k == 0) {
#pragma unroll
          for (int m = 0; m < 9; ++m) pw[P::Y4 + m] = acc4[m];
        }
      }
      if (k == 0) {
        pw[0] = s0;
        pw[1] = s1;
      }
    }
    __syncthreads();
    // combine the waves in a fixed order
    float* nrow = node + size_t(i) * P::NS;
    for (int t = tid; t < P::NS; t += kTeam) {
      float v = part[0][t];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) v += part[w][t];
      nrow[t] = v;
    }
    __syncthreads();
  }
}

template <class P>
int launch(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
           const int64_t* row_ptr, const CompactArgs& ca, float* node, hipStream_t st) {
  int64_t blocks = n < 16384 ? n : 16384;
  if (blocks < 1) return 0;
  if (fidx)
    hipLaunchKernelGGL((forward_kernel<P, true>), dim3(blocks), dim3(kTeam), 0, st, m->dev(), n,
                       fidx, row_ptr, ca, node);
  else
    hipLaunchKernelGGL((forward_kernel<P, false>), dim3(blocks), dim3(kTeam), 0, st, m->dev(), n,
                       species, row_ptr, ca, node);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_forward(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
                   const int64_t* row_ptr, const CompactArgs& ca, float* node, hipStream_t st) {
  const int rc = with_profile(m->C0, m->L, m->R, m->F, [&](auto p, auto) {
    return launch<decltype(p)>(m, n, species, fidx, row_ptr, ca, node, st);
  });
  if (rc == kNoProfile) {
    set_error("forward: profile not compiled");
    return DPA4C_ERR_UNSUPPORTED;
  }
  return rc;
}

}  // namespace dpa4c
