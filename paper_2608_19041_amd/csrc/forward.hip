// Fused forward edge kernel: compaction, featurisation and single
// aggregation.
//
// Methods Eqs. (edge-geometry) .. (moments): for every centre i, the skin
// row is first compacted to the edges inside r_c (compact.h), then those
// edges are scanned once; per edge the envelope, the tabulated radial maps
// g and q, the cached pair coefficients gamma, beta, U, the amplitude psi and
// the harmonics are formed in registers and accumulated into the node state
// [sum chi^2, sum chi^4, Y_lmc].  Apart from the compacted edge records and
// their skin positions, no per-edge quantity is written to memory.
// The readout runs in the per-atom kernel.
//
// Mapping: one wavefront per centre (four centres per 256-thread
// workgroup; the waves never wait for each other).  The wave takes the skin
// row in passes of 64 entries: each lane tests one entry (compact.h), and
// each kept lane forms its edge's per-edge quantities once (envelope, table
// row and offset, harmonics) into the wave's LDS slice.  The lanes then form
// groups of LPE = C1 lanes; each group takes one of the pass's edges at a
// time and lane k of a group owns the channels c = k + LPE*j, so every
// channel c < C1 of the non-scalar degrees sits in slot j = 0.  With folded
// tables a group requests the table entries of its next edge before it
// evaluates the current one.  The groups are combined at the end of the row
// by a fixed xor butterfly, so the node state is the same bits on every run.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "compact.h"
#include "edge_math.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr int kTeam = 256;
constexpr int kWaves = kTeam / kWave;

// Four waves per SIMD fit every degree-three profile without spilling; the
// degree-four one needs more registers per lane.
template <class P>
constexpr int forward_min_waves() { return P::L >= 4 ? 1 : 4; }

template <class P, bool FOLD>
__global__ void __launch_bounds__(kTeam, forward_min_waves<P>()) forward_kernel(ModelDev md, int64_t n,
                                                        const int32_t* __restrict__ typ,
                                                        const int64_t* __restrict__ row_ptr,
                                                        CompactArgs ca,
                                                        float* __restrict__ node) {
  constexpr int G = kWave / P::LPE;   // edge groups in a wave
  // harmonics per edge: u, the degree-two block, then degree three and four
  constexpr int kNH = (3 + 5 + (P::L >= 3 ? 7 : 0) + (P::L >= 4 ? 9 : 0) + 3) / 4 * 4;
  static_assert(P::L < 3 || P::LPE >= (P::L >= 4 ? 9 : 7), "a lane per degree-3/4 component");
  __shared__ float4 pre_all[kWaves][kWave];          // per edge: tau, chi, table row (and pair)
  __shared__ float4 harm_all[kWaves][kWave][kNH / 4];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int grp = lane / P::LPE;
  const int k = lane % P::LPE;
  float4* pre = pre_all[wave];
  float4 (*harm)[kNH / 4] = harm_all[wave];
  const int T1 = md.n_types1;
  const float inv_delta = md.inv_delta;
  const int nf = md.fold_n;
  // ``typ`` holds species (clamped here) or, with folded tables, the folded
  // index of every atom
  auto type_of = [&](int64_t a) { return FOLD ? typ[a] : clamp_type(typ[a], T1); };
  const float w2mask = k < P::C2 ? 1.0f : 0.0f;
  const float w3mask = k < 7 ? 1.0f : 0.0f;
  const float w4mask = k < 9 ? 1.0f : 0.0f;
  const int m3 = k < 7 ? k : 0, m4 = k < 9 ? k : 0;

  for (int64_t blk = xcd_block(blockIdx.x, gridDim.x); blk * kWaves < n; blk += gridDim.x) {
    const int64_t i = blk * kWaves + wave;
    if (i >= n) break;
    const int ai = type_of(i);
    const int64_t b = row_ptr[i];
    int64_t e = row_ptr[i + 1];
    if (b < 0 || e > ca.cap || e < b) e = b;   // malformed row: keep nothing
    const CentreQ ci = centre_q(ca, i);
    float acc0[P::CPL];
#pragma unroll
    for (int j = 0; j < P::CPL; ++j) acc0[j] = 0.0f;
    float acc1[3] = {0.f, 0.f, 0.f};
    float acc2[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
    // degrees three and four have one channel (c = 0): lane k of a group
    // accumulates component m = k of each
    float acc3 = 0.0f, acc4 = 0.0f;
    float s0 = 0.0f, s1 = 0.0f;
    const float* pair_base = FOLD ? md.ftab + size_t(ai) * nf * md.n_rows * (P::C0 * kFoldWords)
                                  : md.pair + size_t(ai) * T1 * (P::C0 * P::PW);

    // One edge's contribution from its LDS entry and, with folded tables,
    // the lane's table entries ``T`` of that edge.
    auto edge_work = [&](int x, const float3* T) {
      const float4 pr = pre[x];
      const float tau = pr.x, chi = pr.y;
      float psi0 = 0.0f;
      if constexpr (FOLD) {
        // the quintic of each channel from the table of the pair (a_i, a_j)
        // (c4 and c5 below float32 resolution, not stored), power form with
        // the float16 c2, c3 scaled through their weights e_n = tau^n / s_n
        // (one mixed-precision FMA each)
        const float t2 = tau * tau, t3 = t2 * tau;
        const float e2 = md.c_inv[0] * t2, e3 = md.c_inv[1] * t3;
#pragma unroll
        for (int jj = 0; jj < P::CPL; ++jj) {
          const uint32_t h23 = __float_as_uint(T[jj].z);
          float psi = fmaf(T[jj].y, tau, T[jj].x);
          psi = fmaf(half_lo(h23), e2, psi);
          psi = fmaf(half_hi(h23), e3, psi);
          acc0[jj] += chi * psi;
          if (jj == 0) psi0 = psi;
        }
      } else {
        const int row = __float_as_int(pr.z), aj = __float_as_int(pr.w);
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
      const float4 ha = harm[x][0], hb = harm[x][1];
      acc1[0] += w * ha.x;
      acc1[1] += w * ha.y;
      acc1[2] += w * ha.z;
      const float w2 = w * w2mask;
      acc2[0] += w2 * ha.w;
      acc2[1] += w2 * hb.x;
      acc2[2] += w2 * hb.y;
      acc2[3] += w2 * hb.z;
      acc2[4] += w2 * hb.w;
      if constexpr (P::L >= 3) {
        // the weight of channel 0 from lane 0 of the group
        const float w0 = __shfl(w, 0, P::LPE);
        const float* he = reinterpret_cast<const float*>(&harm[x][0]);
        acc3 += (w0 * w3mask) * he[8 + m3];
        if constexpr (P::L >= 4) acc4 += (w0 * w4mask) * he[15 + m4];
      }
    };
    // the lane's folded table entries of entry x of the pass
    auto load_rows = [&](int x, float3* T) {
      load_fold_row<P::LPE, P::CPL>(
          pair_base + size_t(__float_as_int(pre[x].z)) * (P::C0 * kFoldWords), k, T);
    };

    int kept = 0;
    for (int64_t s0r = b; s0r < e; s0r += kWave) {
      float4 rec;
      int at;
      const int np = compact_pass(ca, n, b, s0r, e, kept, ci, &rec, &at);
      kept += np;
      // per-edge quantities of the pass's kept edges, in their order; the
      // entries past np get chi = 0, table offset 0 and zero harmonics
      {
        if (at >= 0) {
          float4 pr;
          float hv[kNH];
          const EdgeGeom g = edge_geom(rec.x, rec.y, rec.z);
          float chi, tau;
          envelope(g.rho, md.inv_rc, &chi, nullptr);
          const int row = table_row(g.rho, inv_delta, md.n_rows, &tau);
          const int aj = type_of(__float_as_int(rec.w));
          pr = FOLD ? make_float4(tau, chi, __int_as_float(aj * md.n_rows + row), 0.0f)
                    : make_float4(tau, chi, __int_as_float(row), __int_as_float(aj));
          hv[0] = g.ux;
          hv[1] = g.uy;
          hv[2] = g.uz;
          harm2_h(g.ux, g.uy, g.uz, hv + 3);
          if constexpr (P::L >= 3) harm3_h(g.ux, g.uy, g.uz, hv + 8);
          if constexpr (P::L >= 4) harm4_h(g.ux, g.uy, g.uz, hv + 15);
          pre[at] = pr;
#pragma unroll
          for (int q4 = 0; q4 < kNH / 4; ++q4)
            harm[at][q4] = make_float4(hv[4 * q4], hv[4 * q4 + 1], hv[4 * q4 + 2], hv[4 * q4 + 3]);
        }
        if (lane >= np) {   // at < np <= lane: never the entry a kept lane writes
          pre[lane] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
          for (int q4 = 0; q4 < kNH / 4; ++q4) harm[lane][q4] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      wave_sync();
      if constexpr (FOLD) {
        // the table entries of a group's next edge are requested before its
        // current edge is evaluated (two register sets, used in turn)
        float3 TA[P::CPL], TB[P::CPL];
        if (np > 0) load_rows(grp, TA);
        for (int base = 0; base < np; base += 2 * G) {
          if (base + G < np) load_rows(base + G + grp, TB);
          edge_work(base + grp, TA);
          if (base + G >= np) break;
          if (base + 2 * G < np) load_rows(base + 2 * G + grp, TA);
          edge_work(base + G + grp, TB);
        }
      } else {
        for (int base = 0; base < np; base += G) edge_work(base + grp, nullptr);
      }
      wave_sync();   // the LDS entries are rewritten by the next pass
    }
    if (lane == 0) ca.ecount[i] = kept;

    // combine the groups (fixed xor butterfly over the group index)
#pragma unroll
    for (int off = P::LPE; off < kWave; off <<= 1) {
#pragma unroll
      for (int j = 0; j < P::CPL; ++j) acc0[j] += __shfl_xor(acc0[j], off);
#pragma unroll
      for (int m = 0; m < 3; ++m) acc1[m] += __shfl_xor(acc1[m], off);
#pragma unroll
      for (int m = 0; m < 5; ++m) acc2[m] += __shfl_xor(acc2[m], off);
      if constexpr (P::L >= 3) acc3 += __shfl_xor(acc3, off);
      if constexpr (P::L >= 4) acc4 += __shfl_xor(acc4, off);
      s0 += __shfl_xor(s0, off);
      s1 += __shfl_xor(s1, off);
    }
    if (lane < P::LPE) {
      float* nrow = node + size_t(i) * P::NS;
#pragma unroll
      for (int j = 0; j < P::CPL; ++j) nrow[P::Y0 + j * P::LPE + k] = acc0[j];
#pragma unroll
      for (int m = 0; m < 3; ++m) nrow[P::Y1 + m * P::C1 + k] = acc1[m];
      if (k < P::C2) {
#pragma unroll
        for (int m = 0; m < 5; ++m) nrow[P::Y2 + m * P::C2 + k] = acc2[m];
      }
      if constexpr (P::L >= 3) {
        if (k < 7) nrow[P::Y3 + k] = acc3;
      }
      if constexpr (P::L >= 4) {
        if (k < 9) nrow[P::Y4 + k] = acc4;
      }
      if (k == 0) {
        nrow[0] = s0;
        nrow[1] = s1;
      }
    }
  }
}

template <class P>
int launch(const dpa4c_model* m, int64_t n, const int32_t* species, const int32_t* fidx,
           const int64_t* row_ptr, const CompactArgs& ca, float* node, hipStream_t st) {
  int64_t blocks = (n + kWaves - 1) / kWaves;   // a wave per centre
  blocks = blocks < 65536 ? blocks : 65536;
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
