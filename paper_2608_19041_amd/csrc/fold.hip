// Pair-folded radial tables.
//
// For an ordered type pair (a, b) the amplitude of channel c is a function of
// rho alone (Eq. (amplitude)):
//     psi_c(rho) = gamma_c g_c(rho) + beta_c + sum_mu U_c,mu q_mu(rho).
// Quintic Hermite interpolation is linear in its knot data (value, first and
// second derivative at both ends), and a constant is reproduced exactly, so
// the interpolant of psi_c is gamma_c times the interpolant of g_c, plus
// beta_c, plus U times the interpolants of q (Supplementary Note "Quintic
// Hermite interpolation of the radial table").  Its normalised coefficients
// are that same linear combination of the tabulated ones.
//
// Storage: c0 and c1 in float32, c2 and c3 as float16 scaled by fixed powers
// of two (one per coefficient, from a bound over every pair: |gamma| < 2 and
// |U| < 1 by their tanh forms, times the largest tabulated coefficient); c4
// and c5 are not stored.  With the normalised form c_n Delta^n the
// coefficients fall by about two orders of magnitude per power at
// Delta = 0.002 A, so the whole contribution of c4 and c5 together with the
// 2^-11 relative rounding of c2 and c3 stays below the float32 rounding of
// the value and below 2^-14 of the slope term (checked per model at set-up;
// a model that fails the check runs on the separable float32 tables), and a
// channel takes one 12-byte load instead of 24 bytes.
//
// For the few species of an MD system the library keeps one such table per
// ordered pair present; the edge kernels then read one quintic per channel
// instead of a g quintic, R q quintics and the pair coefficients.  Systems
// with more than kMaxFoldTypes species, or whose folded tables would exceed
// kMaxFoldBytes, use the separable tables directly.  Five species at full
// width (128 channels, 3,000 rows at r_c = 6 A and Delta = 0.002 A) fold into
// 25 tables of 4.6 MB (115 MB, within the last-level cache); on the 5-species
// alloy the folded tables measured faster than the separable ones (backward
// 0.94 -> 0.70 ms at 31,250 atoms, when a folded channel still took 16 B),
// since every edge then reads one 12-byte entry per channel from one table
// instead of 24 B of g coefficients per channel plus the q rows and the pair
// coefficients.
#include <hip/hip_runtime.h>

#include <cstring>
#include <vector>

#include "../../include/dpa4c.h"
#include "edge_math.h"
#include "launch.h"

namespace dpa4c {

namespace {

// species bitmask: each thread collects the bits of its atoms, a wave merges
// them and issues one atomic per word
__global__ void presence_kernel(const int32_t* __restrict__ species, int64_t n, int n_types1,
                                uint32_t* __restrict__ mask) {
  uint32_t m[4] = {0u, 0u, 0u, 0u};
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x) {
    const int a = clamp_type(species[i], n_types1);
    m[a >> 5] |= 1u << (a & 31);
  }
  for (int off = 1; off < kWave; off <<= 1)
    for (int w = 0; w < 4; ++w) m[w] |= __shfl_xor(m[w], off);
  if ((threadIdx.x & (kWave - 1)) == 0)
    for (int w = 0; w < 4; ++w)
      if (m[w]) atomicOr(&mask[w], m[w]);
}

__global__ void fold_index_kernel(const int32_t* __restrict__ species, int64_t n, int n_types1,
                                  const int32_t* __restrict__ map, int32_t* __restrict__ fidx) {
  for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * blockDim.x)
    fidx[i] = map[clamp_type(species[i], n_types1)];
}

struct FoldTypes {
  int t[kMaxFoldTypes];
};

// one block per (table row, folded pair); thread = channel c
__global__ void fold_build_kernel(const float* __restrict__ gtab, const float* __restrict__ qtab,
                                  const float* __restrict__ pair, FoldTypes used, int n_used,
                                  int n_types1, int C0, int R, int LPE, int rows,
                                  const float2 scale, float* __restrict__ ftab) {
  const int s = blockIdx.x, p = blockIdx.y;
  const int a = used.t[p / n_used], b = used.t[p % n_used];
  const int PW = 2 + R, CPL = C0 / LPE;
  for (int c = threadIdx.x; c < C0; c += blockDim.x) {
    const int k = c % LPE, j = c / LPE;
    const float* pc = pair + ((size_t(a * n_types1 + b) * CPL + j) * LPE + k) * PW;
    const float* g = gtab + ((size_t(s) * CPL + j) * LPE + k) * 6;
    // row s of pair p: the (c0, c1) pairs, then the (c2, c3) words, each
    // permuted so that lane k's values for its channels are adjacent (the
    // order the edge kernels read, load_fold_row)
    float* row = ftab + (size_t(p) * rows + s) * C0 * kFoldWords;
    float* pr = row + ((j / 2) * LPE + k) * 4 + 2 * (j % 2);
    uint32_t* wd = reinterpret_cast<uint32_t*>(row + 2 * C0) +
                   (CPL == 2 ? 2 * k + j : ((j / 4) * LPE + k) * 4 + j % 4);
    double v[4];
    for (int q = 0; q < 4; ++q) {
      v[q] = double(pc[0]) * double(g[q]) + (q == 0 ? double(pc[1]) : 0.0);
      for (int mu = 0; mu < R; ++mu)
        v[q] += double(pc[2 + mu]) * double(qtab[(size_t(s) * R + mu) * 6 + q]);
    }
    const float sc[2] = {scale.x, scale.y};
    uint16_t hb[2];
    for (int q = 0; q < 2; ++q)
      hb[q] = __builtin_bit_cast(uint16_t,
                                 static_cast<_Float16>(static_cast<float>(v[2 + q] * sc[q])));
    pr[0] = static_cast<float>(v[0]);
    pr[1] = static_cast<float>(v[1]);
    *wd = uint32_t(hb[0]) | (uint32_t(hb[1]) << 16);
  }
}

__global__ void zero_u32_kernel(uint32_t* p, int n) {
  if (static_cast<int>(threadIdx.x) < n) p[threadIdx.x] = 0u;
}

int grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  return static_cast<int>(b < 4096 ? (b < 1 ? 1 : b) : 4096);
}

}  // namespace

int prepare_species(dpa4c_model* m, const int32_t* species, int64_t n, uint32_t* mask_dev,
                    int32_t* fidx, bool may_alloc, bool* use_fold, hipStream_t st) {
  Workspace& w = m->ws;
  const int T1 = m->n_types + 1;
  *use_fold = false;
  if (n <= 0) return 0;
  // the type map and the pinned host words ([0, 16) the presence mask,
  // [64, 64 + 4 T1) the type map) are allocated with the model
  if (!w.fold_host || !w.fold_map.p) {
    set_error("prepare_species: the model's species buffers are missing");
    return DPA4C_ERR_INVALID_ARG;
  }
  hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(64), 0, st, mask_dev, 4);
  hipLaunchKernelGGL(presence_kernel, dim3(grid_for(n)), dim3(256), 0, st, species, n, T1, mask_dev);
  DPA4C_HIP_TRY(hipGetLastError());
  DPA4C_HIP_TRY(hipMemcpyAsync(w.fold_host, mask_dev, 4 * sizeof(uint32_t), hipMemcpyDeviceToHost,
                               st));
  DPA4C_HIP_TRY(hipStreamSynchronize(st));
  uint32_t mask[4];
  std::memcpy(mask, w.fold_host, sizeof(mask));
  const bool same = m->fold_n >= 0 && std::memcmp(mask, m->fold_types_mask, sizeof(mask)) == 0;
  if (!same) {
    FoldTypes used{};
    int n_used = 0;
    std::vector<int32_t> map(T1, -1);
    for (int a = 0; a < T1; ++a)
      if (mask[a >> 5] >> (a & 31) & 1u) {
        if (n_used < kMaxFoldTypes) {
          used.t[n_used] = a;
          map[a] = n_used;
        }
        ++n_used;
      }
    const size_t per_pair = size_t(m->n_rows) * m->C0 * kFoldWords;
    const size_t need = 4 * per_pair * size_t(n_used) * size_t(n_used);
    if (!m->fold_allowed || n_used > kMaxFoldTypes || need > kMaxFoldBytes) {
      std::memcpy(m->fold_types_mask, mask, sizeof(mask));
      m->fold_n = 0;   // the separable tables are used
    } else if (!may_alloc && need > w.ftab.bytes) {
      return 0;        // this call only: separable tables, the folded state kept
    } else {
      DPA4C_TRY(w.ftab.ensure(need));
      std::memcpy(m->fold_types_mask, mask, sizeof(mask));
      int32_t* hmap = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(w.fold_host) + 64);
      std::memcpy(hmap, map.data(), 4 * size_t(T1));
      DPA4C_HIP_TRY(hipMemcpyAsync(w.fold_map.p, hmap, 4 * size_t(T1), hipMemcpyHostToDevice, st));
      hipLaunchKernelGGL(fold_build_kernel, dim3(m->n_rows, n_used * n_used),
                         dim3(m->C0 < 256 ? m->C0 : 256), 0, st, m->gtab, m->qtab, m->pair, used,
                         n_used, T1, m->C0, m->R, m->C[1], m->n_rows,
                         make_float2(m->c_scale[0], m->c_scale[1]),
                         w.ftab.as<float>());
      DPA4C_HIP_TRY(hipGetLastError());
      m->fold_n = n_used;
    }
  }
  if (m->fold_n > 0) {
    hipLaunchKernelGGL(fold_index_kernel, dim3(grid_for(n)), dim3(256), 0, st, species, n, T1,
                       w.fold_map.as<int32_t>(), fidx);
    DPA4C_HIP_TRY(hipGetLastError());
    *use_fold = true;
  }
  return 0;
}

}  // namespace dpa4c
