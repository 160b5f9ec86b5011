// Per-atom kernel: readout, atomic-energy MLP, head, MLP input gradient and
// readout vector-Jacobian product for a tile of 16 atoms in one workgroup
// (Eqs. (alignment) .. (fitting)).  The descriptor D and dE/dD never leave
// LDS: the node state Y comes in, E_i and dE/d(node state) go out.
//
//   h1 = SiLU(D Th1 + b1), h2 = SiLU(h1 Th2 + b2) + h1, h3 = SiLU(h2 Th3 + b3) + h2
//   E  = h3 . w + b + E_ref[a]
//   hb2 = w + (w * s3) Th3^T,  hb1 = hb2 + (hb2 * s2) Th2^T,  dE/dD = (hb1 * s1) Th1^T
// with s_t = SiLU'(pre_t).  Every product runs on v_mfma_f32_16x16x4_f32.
//
// Layout: the 16-row activation tile (the A operand) lives in LDS; each of the
// eight waves owns a fixed set of 16-column output tiles, so the SiLU'
// factors and the residual carry of every (row, column) stay in the same
// lane's registers from the forward to the backward pass.  Weights are
// stored in fragment order: for output tile T and k-block kb (16 inputs) lane
// l reads one float4 = W[kb*16 + 4*(l/16) + s][T*16 + l%16], s = 0..3, and
// the A operand uses the same permutation of k inside the block.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "launch.h"
#include "readout.h"

namespace dpa4c {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kRows = 16;
constexpr int kThreads = 512;
constexpr int kWavesPB = kThreads / 64;

// logistic function with the hardware reciprocal (v_rcp_f32, within 1 ulp):
// the epilogues between products take 36 of them per lane and tile, and the
// correctly rounded division would cost about ten instructions each
__device__ inline float sigm(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// One 16-byte load through a buffer resource: descriptor and tile offset in
// scalar registers, only the lane offset in a vector register (no per-lane
// 64-bit addresses to keep alive; reads past the resource return zero).
typedef unsigned u4 __attribute__((ext_vector_type(4)));
constexpr int kBufWord3 = 0x00020000;   // raw 32-bit buffer, gfx9 data format

__device__ inline float4 buf_load16(__amdgpu_buffer_rsrc_t rs, unsigned voff, int soff) {
  const u4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(voff), soff, 0);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}

// B operand stream of one product: the weight resource, the byte offset of
// each of the wave's output tiles and the first two k-blocks, which do not
// depend on the A tile and so are requested before the barrier that
// publishes it (by the drain of the previous product).  Tiles past
// ``ntiles`` repeat the last tile; ``first`` must be wave-uniform.
template <int MAXT>
struct BStream {
  __amdgpu_buffer_rsrc_t rs;
  int toff[MAXT];
  float4 b0[MAXT], b1[MAXT];
};

template <int MAXT>
__device__ inline void bstream_open(BStream<MAXT>& bs, const float4* __restrict__ Wf, int kblocks,
                                    int first, int stride, int ntiles, unsigned lane16) {
  bs.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float4*>(Wf), 0, ntiles * kblocks * 1024,
                                            kBufWord3);
#pragma unroll
  for (int t = 0; t < MAXT; ++t) {
    const int T = first + t * stride < ntiles ? first + t * stride : ntiles - 1;
    bs.toff[t] = T * kblocks * 1024;
  }
#pragma unroll
  for (int t = 0; t < MAXT; ++t) bs.b0[t] = buf_load16(bs.rs, lane16, bs.toff[t]);
#pragma unroll
  for (int t = 0; t < MAXT; ++t)
    bs.b1[t] = buf_load16(bs.rs, lane16, bs.toff[t] + (kblocks > 1 ? 1024 : 0));
}

// acc[t] += A (16 x K, LDS, row stride lda) * W (fragment order) for the
// first NT tiles of ``bs`` (NT <= MAXT).  Three k-blocks of B and A are in
// flight: k-block kb+2 is requested before the MFMAs of kb start, and the
// MFMAs of one k-block are interleaved across tiles so that consecutive
// instructions do not depend on each other.  No load runs past the last
// k-block; ``drain()`` is called once the last one is requested, so the
// caller can start the loads of what follows the product.
template <int NT, int MAXT, class Drain>
__device__ inline void mfma_tiles(v4f* acc, const float* __restrict__ As, int lda, int kblocks,
                                  BStream<MAXT>& bs, unsigned lane, unsigned lane16,
                                  Drain&& drain) {
  static_assert(NT <= MAXT, "tile count");
  const float* ap = As + (lane & 15) * lda + (lane >> 4) * 4;
  auto step = [&](const float4& a, const float4* b) {
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b[t].x, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b[t].y, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b[t].z, acc[t], 0, 0, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b[t].w, acc[t], 0, 0, 0);
  };
  auto ld_b = [&](float4* b, int kk) {
#pragma unroll
    for (int t = 0; t < NT; ++t) b[t] = buf_load16(bs.rs, lane16, bs.toff[t] + kk * 1024);
  };
  auto ld_a = [&](int kk) { return *reinterpret_cast<const float4*>(ap + kk * 16); };
  float4* b0 = bs.b0;
  float4* b1 = bs.b1;
  float4 b2[NT];
  float4 a0 = ld_a(0), a1 = ld_a(kblocks > 1 ? 1 : 0), a2;
  int kb = 0;
#pragma unroll 1
  for (; kb + 5 <= kblocks; kb += 3) {
    ld_b(b2, kb + 2);
    a2 = ld_a(kb + 2);
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch ahead of the MFMAs
    step(a0, b0);
    ld_b(b0, kb + 3);
    a0 = ld_a(kb + 3);
    __builtin_amdgcn_sched_barrier(0);
    step(a1, b1);
    ld_b(b1, kb + 4);
    a1 = ld_a(kb + 4);
    __builtin_amdgcn_sched_barrier(0);
    step(a2, b2);
  }
  // the last two to four k-blocks; kb and kb + 1 are already in b0/a0, b1/a1
  const int rem = kblocks - kb;
  if (rem >= 3) {
    ld_b(b2, kb + 2);
    a2 = ld_a(kb + 2);
  }
  if (rem <= 3) drain();
  __builtin_amdgcn_sched_barrier(0);
  step(a0, b0);
  if (rem == 4) {
    ld_b(b0, kb + 3);
    a0 = ld_a(kb + 3);
    drain();
  }
  __builtin_amdgcn_sched_barrier(0);
  if (rem >= 2) step(a1, b1);
  if (rem >= 3) step(a2, b2);
  if (rem == 4) step(a0, b0);
}

struct MlpArgs {
  const float4* W[3];     // forward weights, fragment order (K = Kp, F, F; N = F)
  const float4* WT[3];    // transposed weights, fragment order (K = F; N = F, F, Kp)
  const float* bias[3];
  const float* w_head;
  float b_head;
  const float* E_ref;
  int n_types1;
};

// P: model profile (KP = P::DSTR padded descriptor width), F: hidden width.
template <class P, int F>
__global__ void __launch_bounds__(kThreads) atom_kernel(MlpArgs p, ModelDev md, int64_t n,
                                                        const int32_t* __restrict__ species,
                                                        const float* __restrict__ node,
                                                        float* __restrict__ node_grad,
                                                        double* __restrict__ e_atom,
                                                        float* __restrict__ desc_out) {
  constexpr int KP = P::DSTR;
  constexpr int LDA = (KP > F ? KP : F) + 4;
  constexpr int FT = F / 16;                          // output tiles of a hidden layer
  constexpr int NT = (FT + kWavesPB - 1) / kWavesPB;  // per wave (round-robin)
  constexpr int DT = KP / 16;                         // output tiles of dE/dD
  constexpr int NTD = (DT + kWavesPB - 1) / kWavesPB;
  constexpr int NTD1 = NTD > 1 ? NTD - 1 : 1;         // the shorter dE/dD product
  constexpr int APW = kRows / kWavesPB;               // atoms per wave in the readouts
  // Two activation tiles: a product reads one and its epilogue writes the
  // other, so a wave that has finished its share of a product goes on to its
  // epilogue while the others still read (one barrier per layer).  As (row
  // stride LDA) holds D, h2, p3, p1 and dE/dD; Bs (LDB) holds h1 and p2.
  // Only where the workgroup already has a CU to itself and the second tile
  // still fits in LDS; otherwise both are As, with a barrier between a
  // product and its epilogue.
  constexpr int LDB = F + 4;
  constexpr size_t kBase = sizeof(float) * kRows * LDA + sizeof(ReadoutLds<P>) * kRows +
                           sizeof(ReadoutParams<P>) + sizeof(float) * kWavesPB * kRows;
  constexpr bool kTwo =
      kBase > 80 * 1024 && kBase + sizeof(float) * kRows * LDB + 1024 <= 160 * 1024;
  __shared__ float As[kRows * LDA];
  __shared__ float Bs_buf[kTwo ? kRows * LDB : 1];
  float* const Bs = kTwo ? Bs_buf : As;
  constexpr int LDBv = kTwo ? LDB : LDA;
  __shared__ float epart[kWavesPB][kRows];
  __shared__ ReadoutLds<P> rl_all[kRows];   // one per atom of the tile
  __shared__ ReadoutParams<P> rp;
  // wave index made visibly uniform, so per-wave addresses stay scalar
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col_in = lane & 15, rgrp = lane >> 4;   // output element: row 4*rgrp + r
  const unsigned lane16 = 16u * lane;               // byte offset of a lane's fragment
  const int nt = (FT - wave + kWavesPB - 1) / kWavesPB;
  static_assert(APW == 2, "a wave reads out two atoms, one per half");
  const int half = lane >> 5, hl = lane & 31;
  const int ra = wave * APW + half;         // tile row of this half-wave's atom
  // the same objects seen through LDS-address-space pointers (C-style casts:
  // an address-space conversion)
  DPA4C_LDS ReadoutLds<P>& rl = *(DPA4C_LDS ReadoutLds<P>*)(&rl_all[ra]);
  const DPA4C_LDS ReadoutParams<P>& rpl = *(DPA4C_LDS ReadoutParams<P>*)(&rp);
  DPA4C_LDS float* arow = (DPA4C_LDS float*)(As + ra * LDA);
  stage_readout_params<P>(rp, md, threadIdx.x, kThreads);
  // The half-wave's share of its atom's node state (zero past n) and the
  // atom's species, requested one tile ahead: the loads for the next tile are
  // issued after the current tile's readout and complete during its MLP.
  constexpr int NY = (P::NS + kHalf - 1) / kHalf;
  float ynext[NY];
  int snext = 0;
  auto fetch_node = [&](int64_t tl) {
    const int64_t i = tl * kRows + ra;
    const bool ok = i < n;
    const float* ny = node + size_t(ok ? i : 0) * P::NS;
#pragma unroll
    for (int q = 0; q < NY; ++q) {
      const int t = hl + q * kHalf;
      ynext[q] = (ok && t < P::NS) ? ny[t] : 0.0f;
    }
    snext = ok ? species[i] : 0;
  };
  fetch_node(blockIdx.x);
  __syncthreads();

  for (int64_t tile = blockIdx.x; tile * kRows < n; tile += gridDim.x) {
    const int64_t row0 = tile * kRows;
    // ---- readout of the tile's atoms: D rows into LDS (rows past n get
    // a zero node state and are zeroed afterwards)
    {
      const int64_t i = row0 + ra;
      const bool ok = i < n;
#pragma unroll
      for (int q = 0; q < NY; ++q) {
        const int t = hl + q * kHalf;
        if (t < P::NS) rl.y[t] = ynext[q];
      }
      const float* x0 = md.type_embed + size_t(ok ? clamp_type(snext, md.n_types1) : 0) * P::C0;
      wave_sync();
      readout_forward<P>(rl, rpl, x0, arow);
      if (ok && desc_out)
        for (int t = hl; t < P::DOUT; t += kHalf) desc_out[size_t(i) * P::DOUT + t] = arow[t];
      if (!ok)
        for (int t = hl; t < KP; t += kHalf) arow[t] = 0.0f;
    }
    BStream<NT> bs;    // the B stream of the next hidden-width product
    bstream_open(bs, p.W[0], KP / 16, wave, kWavesPB, FT, lane16);
    fetch_node(tile + gridDim.x);
    __syncthreads();

    float s[3][NT][4];   // SiLU'(pre) of the three layers
    float h[NT][4];      // current activation / backward carry
    float wh[NT];        // head weights of the wave's columns
#pragma unroll
    for (int layer = 0; layer < 3; ++layer) {
      // layer 0 reads D from As and writes h1 to Bs, layer 1 reads Bs and
      // writes h2 to As, layer 2 reads As; h3 stays in registers (head)
      const float* src = layer == 1 ? Bs : As;
      const int lds = layer == 1 ? LDBv : LDA;
      float* dst = layer == 0 ? Bs : As;
      const int ldd = layer == 0 ? LDBv : LDA;
      v4f acc[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};
      float bias[NT];
      BStream<NT> bsn;
      mfma_tiles<NT>(acc, src, lds, (layer == 0 ? KP : F) / 16, bs, lane, lane16, [&] {
#pragma unroll
        for (int t = 0; t < NT; ++t)
          bias[t] = t < nt ? p.bias[layer][(wave + kWavesPB * t) * 16 + col_in] : 0.0f;
        if (layer < 2) {
          bstream_open(bsn, p.W[layer + 1], F / 16, wave, kWavesPB, FT, lane16);
        } else {
#pragma unroll
          for (int t = 0; t < NT; ++t)
            wh[t] = t < nt ? p.w_head[(wave + kWavesPB * t) * 16 + col_in] : 0.0f;
          bstream_open(bsn, p.WT[2], F / 16, wave, kWavesPB, FT, lane16);
        }
      });
      bs = bsn;
      if constexpr (!kTwo) __syncthreads();   // everyone has read the A tile
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= nt) continue;
        const int col = (wave + kWavesPB * t) * 16 + col_in;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pre = acc[t][r] + bias[t];
          const float sg = sigm(pre);
          const float act = pre * sg;
          s[layer][t][r] = sg * (1.0f + pre * (1.0f - sg));
          h[t][r] = layer == 0 ? act : act + h[t][r];   // identity residual for equal widths
          if (layer < 2) dst[(4 * rgrp + r) * ldd + col] = h[t][r];
        }
      }
      __syncthreads();   // the next A tile is complete, and this one is read
    }
    // ---- head: E_i = h3 . w + b + E_ref, fixed-order reduction
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t >= nt) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) part[r] += h[t][r] * wh[t];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) part[r] += __shfl_xor(part[r], off, 16);
    }
    if (col_in == 0) {
#pragma unroll
      for (int r = 0; r < 4; ++r) epart[wave][4 * rgrp + r] = part[r];
    }
    // ---- backward seed: hbar3 = w, p3 = w * s3 as the next A operand
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t >= nt) continue;
      const int col = (wave + kWavesPB * t) * 16 + col_in;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        h[t][r] = wh[t];                                // carry hbar3
        As[(4 * rgrp + r) * LDA + col] = wh[t] * s[2][t][r];
      }
    }
    __syncthreads();
    if (threadIdx.x < kRows && row0 + threadIdx.x < n) {
      const int i = static_cast<int>(threadIdx.x);
      float e = epart[0][i];
#pragma unroll
      for (int w = 1; w < kWavesPB; ++w) e += epart[w][i];
      int a = species[row0 + i];
      a = static_cast<unsigned>(a) < static_cast<unsigned>(p.n_types1) ? a : p.n_types1 - 1;
      e_atom[row0 + i] = double(e) + double(p.b_head) + double(p.E_ref[a]);
    }
    // ---- hbar_{t-1} = hbar_t + p_t Th_t^T,  p_{t-1} = hbar_{t-1} * s_{t-1}
    BStream<NTD> bsd;   // the B stream of dE/dD
#pragma unroll
    for (int layer = 2; layer >= 1; --layer) {
      // layer 2 reads p3 from As and writes p2 to Bs, layer 1 reads Bs and
      // writes p1 to As
      const float* src = layer == 2 ? As : Bs;
      const int lds = layer == 2 ? LDA : LDBv;
      float* dst = layer == 2 ? Bs : As;
      const int ldd = layer == 2 ? LDBv : LDA;
      v4f acc[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};
      BStream<NT> bsn;
      mfma_tiles<NT>(acc, src, lds, F / 16, bs, lane, lane16, [&] {
        if (layer == 2)
          bstream_open(bsn, p.WT[1], F / 16, wave, kWavesPB, FT, lane16);
        else
          bstream_open(bsd, p.WT[0], F / 16, wave, kWavesPB, DT, lane16);
      });
      if (layer == 2) bs = bsn;
      if constexpr (!kTwo) __syncthreads();   // everyone has read the A tile
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= nt) continue;
        const int col = (wave + kWavesPB * t) * 16 + col_in;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          h[t][r] += acc[t][r];
          dst[(4 * rgrp + r) * ldd + col] = h[t][r] * s[layer - 1][t][r];
        }
      }
      __syncthreads();
    }
    // ---- dE/dD = p1 Th1^T  (KP columns, tiles dealt round-robin) back into LDS,
    // divided by the calibration scales; a wave with one tile fewer runs the
    // shorter product
    {
      const int ntd = (DT - wave + kWavesPB - 1) / kWavesPB;
      v4f acc[NTD];
#pragma unroll
      for (int t = 0; t < NTD; ++t) acc[t] = v4f{0.f, 0.f, 0.f, 0.f};
      if (ntd == NTD)
        mfma_tiles<NTD>(acc, As, LDA, F / 16, bsd, lane, lane16, [] {});
      else
        mfma_tiles<NTD1>(acc, As, LDA, F / 16, bsd, lane, lane16, [] {});
      __syncthreads();
#pragma unroll
      for (int t = 0; t < NTD; ++t) {
        if (t >= ntd) continue;
        const int col = (wave + kWavesPB * t) * 16 + col_in;
        const float is = rpl.inv_sigma[col];   // dE/dD~ = dE/dD / sigma, Eq. (calibration)
#pragma unroll
        for (int r = 0; r < 4; ++r) As[(4 * rgrp + r) * LDA + col] = acc[t][r] * is;
      }
      __syncthreads();
    }
    // ---- readout VJP: dE/d(node state) of the tile's atoms, from the
    // forward intermediates still held in rl
    {
      const int64_t i = row0 + ra;
      readout_backward<P>(rl, rpl, arow);
      if (i < n) {
        float* gout = node_grad + size_t(i) * P::NS;
        for (int t = hl; t < P::NS; t += kHalf) gout[t] = rl.gy[t];
      }
    }
    __syncthreads();
  }
}

template <class P, int F>
int launch_atoms(const dpa4c_model* m, int64_t n, const int32_t* species, const float* node,
                 float* node_grad, double* e_atom, float* desc_out, hipStream_t st) {
  MlpArgs a{};
  for (int t = 0; t < 3; ++t) {
    a.W[t] = reinterpret_cast<const float4*>(m->wfrag[t]);
    a.WT[t] = reinterpret_cast<const float4*>(m->wfragT[t]);
    a.bias[t] = m->bias[t];
  }
  a.w_head = m->w_head;
  a.b_head = m->b_head;
  a.E_ref = m->E_ref;
  a.n_types1 = m->n_types + 1;
  int64_t tiles = (n + kRows - 1) / kRows;
  int64_t grid = tiles < 16384 ? tiles : 16384;
  if (grid < 1) grid = 1;
  hipLaunchKernelGGL((atom_kernel<P, F>), dim3(grid), dim3(kThreads), 0, st, a, m->dev(), n,
                     species, node, node_grad, e_atom, desc_out);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_atoms(const dpa4c_model* m, int64_t n, const int32_t* species, const float* node,
                 float* node_grad, double* e_atom, float* desc_out, hipStream_t st) {
  if (n <= 0) return 0;
  if (m->n_layers != 3 || !m->wfrag[0]) {
    set_error("the per-atom kernel needs three hidden layers");
    return DPA4C_ERR_UNSUPPORTED;
  }
  const int rc = with_profile(m->C0, m->L, m->R, m->F, [&](auto p, auto f) {
    return launch_atoms<decltype(p), decltype(f)::value>(m, n, species, node, node_grad, e_atom,
                                                         desc_out, st);
  });
  if (rc != kNoProfile) return rc;
  set_error("no per-atom kernel instance for this (profile, MLP width)");
  return DPA4C_ERR_UNSUPPORTED;
}

}  // namespace dpa4c
