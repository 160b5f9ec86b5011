// Per-row compaction of the skin list to the edges inside r_c (Eq.
// (neighbor-set) with the fixed-point predicate of the neighbour builder),
// done by the workgroup that then evaluates the row.
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
  const int32_t* skin_rev;    // [cap] position of the reverse of each skin edge in row j
  int32_t* cidx;              // [cap] out: compact slot of each skin edge, or -1, counted
                              // from the head of its row
  int32_t* crev;              // [cap] out: skin_rev of the skin edge of each compact slot
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

// Keeps the skin edges of row i inside r_c, in canonical order, and writes
// their records r_ij = (r_j + sum_b n_b h_b) - r_i (float64 difference stored as
// float32) to the first slots of the row, and for every skin edge its
// row-local compact slot (or -1) and, per compact slot, the reverse position
// of its skin edge.  All TEAM threads of the
// workgroup take part; ``wtot`` is LDS scratch of TEAM/64 ints.  Returns
// the number kept (the same in every thread); the records are visible to
// the whole workgroup on return.
template <int TEAM>
__device__ inline int compact_row(const CompactArgs& a, int64_t n, int64_t i, int64_t b, int64_t e,
                                  int* wtot) {
  constexpr int W = TEAM / kWave;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const double xi = a.pos[3 * i], yi = a.pos[3 * i + 1], zi = a.pos[3 * i + 2];
  const int64_t qi0 = qfix_dev(xi), qi1 = qfix_dev(yi), qi2 = qfix_dev(zi);
  if (b < 0 || e > a.cap || e < b) e = b;   // malformed row: keep nothing
  int kept = 0;
  for (int64_t base = b; base < e; base += TEAM) {
    const int64_t s = base + tid;
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
        int64_t dx = qfix_dev(xj) - qi0, dy = qfix_dev(yj) - qi1, dz = qfix_dev(zj) - qi2;
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
    if (lane == 0) wtot[wave] = __popcll(m);
    __syncthreads();
    int off = 0, total = 0;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const int c = wtot[w];
      off += w < wave ? c : 0;
      total += c;
    }
    if (s < e) {
      if (pred) {
        const int slot = kept + off + pre;
        double rx, ry, rz;
        if (!a.tric) {
          rx = (xj + nx * a.h[0]) - xi;
          ry = (yj + ny * a.h[4]) - yi;
          rz = (zj + nz * a.h[8]) - zi;
        } else {   // (r_j + sum_b n_b h_b) - r_i
          rx = (xj + (nx * a.h[0] + ny * a.h[3] + nz * a.h[6])) - xi;
          ry = (yj + (nx * a.h[1] + ny * a.h[4] + nz * a.h[7])) - yi;
          rz = (zj + (nx * a.h[2] + ny * a.h[5] + nz * a.h[8])) - zi;
        }
        a.edge[b + slot] = make_float4(static_cast<float>(rx), static_cast<float>(ry),
                                   static_cast<float>(rz), __int_as_float(j));
        a.cidx[s] = slot;
        a.crev[b + slot] = a.skin_rev[s];
      } else {
        a.cidx[s] = -1;
      }
    }
    kept += total;
    __syncthreads();   // wtot is reused; the records are written
  }
  if (tid == 0) a.ecount[i] = kept;
  return kept;
}

}  // namespace dpa4c
