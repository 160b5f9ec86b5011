// Per-row compaction of the skin list to the edges inside r_c (Eq.
// (neighbor-set) with the fixed-point predicate of the neighbour builder),
// done by the wavefront that then evaluates the row.
#pragma once

#include "common.h"
#include "edge_math.h"

namespace dpa4c {

// inputs and outputs of the compaction (one struct, passed by value)
struct CompactArgs {
  const double* pos;          // [N][3]
  const int32_t* nbr_j;       // skin list
  const int32_t* nbr_shift;
  int64_t qh[9];              // lattice vectors, fixed point, row b = Q(h_b)
  int64_t rcq;                // cutoff, fixed point
  double h[9];                // lattice vectors (A), row b = h_b
  int tric;                   // 0: diagonal cell (only h_00, h_11, h_22 are used)
  int64_t cap;                // skin-list capacity
  int32_t* ecount;            // [N] out: edges kept per row
  float4* edge;               // [cap] out: (r_ij, bits of j) at the head of each skin row
  int32_t* cskin;             // [cap] out: for each compact slot of a row, the position of
                              // its skin entry in the row (both counted from the row's head)
};

__device__ inline int64_t qfix_dev(double x) {
  return static_cast<int64_t>(__builtin_rint(x * kQScale));
}

// strictly within the fixed-point radius; components are rejected before
// squaring, so nothing overflows
__device__ inline bool within_q(int64_t dx, int64_t dy, int64_t dz, int64_t rq) {
  if (dx >= rq || dx <= -rq || dy >= rq || dy <= -rq || dz >= rq || dz <= -rq) return false;
  return dx * dx + dy * dy + dz * dz < rq * rq;
}

// Fixed-point position of a centre, read once per row.
struct CentreQ {
  double x, y, z;
  int64_t q0, q1, q2;
};
// ``i`` is the same in every lane of the wave; the values are moved to
// scalar registers, which keeps them out of the vector register budget.
__device__ inline int64_t wave_uniform(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32));
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}
__device__ inline double wave_uniform(double v) {
  return __builtin_bit_cast(double, wave_uniform(__builtin_bit_cast(int64_t, v)));
}
__device__ inline CentreQ centre_q(const CompactArgs& a, int64_t i) {
  CentreQ c;
  c.x = wave_uniform(a.pos[3 * i]);
  c.y = wave_uniform(a.pos[3 * i + 1]);
  c.z = wave_uniform(a.pos[3 * i + 2]);
  c.q0 = wave_uniform(qfix_dev(c.x));
  c.q1 = wave_uniform(qfix_dev(c.y));
  c.q2 = wave_uniform(qfix_dev(c.z));
  return c;
}

// One pass of a wavefront over the skin entries [s0, s0 + 64) of the row
// [b, e) of centre ``ci``: lane l tests entry s0 + l with the exact predicate,
// and the entries inside r_c keep canonical order.  ``kept`` edges of the row
// precede the pass.  A kept lane writes its record r_ij = (r_j + sum_b n_b
// h_b) - r_i (float64 difference stored as float32) to compact slot kept +
// *at of the row, and the position of its skin entry in the row to the same
// slot of cskin; it returns the record in *rec and its rank within the pass
// in *at (-1 for lanes that keep nothing).  Returns the number kept
// by the pass (the same in every lane).
__device__ inline int compact_pass(const CompactArgs& a, int64_t n, int64_t b, int64_t s0,
                                   int64_t e, int kept, const CentreQ& ci, float4* rec, int* at) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t s = s0 + lane;
  bool pred = false;
  int32_t j = 0;
  int nx = 0, ny = 0, nz = 0;
  double xj = 0.0, yj = 0.0, zj = 0.0;   // kept for the record (one gather each)
  if (s < e) {
    j = a.nbr_j[s];
    const int32_t sh = a.nbr_shift[s];
    nx = unpack_x(sh);
    ny = unpack_y(sh);
    nz = unpack_z(sh);
    if (j >= 0 && j < n) {
      xj = a.pos[3 * j];
      yj = a.pos[3 * j + 1];
      zj = a.pos[3 * j + 2];
      int64_t dx = qfix_dev(xj) - ci.q0, dy = qfix_dev(yj) - ci.q1, dz = qfix_dev(zj) - ci.q2;
      if (!a.tric) {
        dx += nx * a.qh[0];
        dy += ny * a.qh[4];
        dz += nz * a.qh[8];
      } else {   // sum_b n_b Q(h_b)
        dx += nx * a.qh[0] + ny * a.qh[3] + nz * a.qh[6];
        dy += nx * a.qh[1] + ny * a.qh[4] + nz * a.qh[7];
        dz += nx * a.qh[2] + ny * a.qh[5] + nz * a.qh[8];
      }
      pred = within_q(dx, dy, dz, a.rcq);
    }
  }
  const uint64_t m = __ballot(pred);
  const int pre = __popcll(m & ((uint64_t(1) << lane) - 1));
  *at = -1;
  if (s < e) {
    if (pred) {
      const int slot = kept + pre;
      double rx, ry, rz;
      if (!a.tric) {
        rx = (xj + nx * a.h[0]) - ci.x;
        ry = (yj + ny * a.h[4]) - ci.y;
        rz = (zj + nz * a.h[8]) - ci.z;
      } else {   // (r_j + sum_b n_b h_b) - r_i
        rx = (xj + (nx * a.h[0] + ny * a.h[3] + nz * a.h[6])) - ci.x;
        ry = (yj + (nx * a.h[1] + ny * a.h[4] + nz * a.h[7])) - ci.y;
        rz = (zj + (nx * a.h[2] + ny * a.h[5] + nz * a.h[8])) - ci.z;
      }
      *rec = make_float4(static_cast<float>(rx), static_cast<float>(ry), static_cast<float>(rz),
                         __int_as_float(j));
      a.edge[b + slot] = *rec;
      a.cskin[b + slot] = static_cast<int32_t>(s - b);
      *at = pre;
    }
  }
  return __popcll(m);
}

}  // namespace dpa4c
