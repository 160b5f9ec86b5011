// Force assembly, energy reduction and velocity-Verlet kernels.
//
// Forces, Eq. (forces): F_k = sum_{j in N_k} dE/dr_kj - sum_{i: k in N_i} dE/dr_ik.
// Every edge e = (k -> j, n) of row k has a reverse edge rev(e) = (j -> k, -n)
// in row j, so F_k = sum over row k of (g_e - g_rev(e)): one reduction per
// atom over its own row, in a fixed order, in float64, with no atomics.
// The total energy is a fixed-order two-pass float64 sum.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr int kBlock = 256;
constexpr int kLanesPerAtom = 16;
constexpr int kRedBlock = 256;
constexpr int kRedPer = 16;                 // elements per thread in the first pass

// first pass: block b sums the fixed slice [b*T, (b+1)*T) of x (times w if
// given), in a fixed tree order
__device__ inline double block_sum(double v, double* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int off = kRedBlock / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) sh[threadIdx.x] += sh[threadIdx.x + off];
    __syncthreads();
  }
  return sh[0];
}

__global__ void __launch_bounds__(kRedBlock) partial_sum_kernel(const double* __restrict__ x, int64_t n,
                                                                double* __restrict__ partials) {
  __shared__ double sh[kRedBlock];
  const int64_t base = blockIdx.x * int64_t(kRedBlock * kRedPer) + threadIdx.x;
  double s = 0.0;
  for (int t = 0; t < kRedPer; ++t) {
    int64_t i = base + int64_t(t) * kRedBlock;
    if (i < n) s += x[i];
  }
  double tot = block_sum(s, sh);
  if (threadIdx.x == 0) partials[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(kRedBlock) final_sum_kernel(const double* __restrict__ partials,
                                                              int64_t np, double* __restrict__ out) {
  __shared__ double sh[kRedBlock];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < np; i += kRedBlock) s += partials[i];
  double tot = block_sum(s, sh);
  if (threadIdx.x == 0) *out = tot;
}

int fixed_sum(const double* x, int64_t n, double* partials, double* out, hipStream_t st) {
  int64_t np = (n + kRedBlock * kRedPer - 1) / (kRedBlock * kRedPer);
  if (np < 1) np = 1;
  hipLaunchKernelGGL(partial_sum_kernel, dim3(np), dim3(kRedBlock), 0, st, x, n, partials);
  hipLaunchKernelGGL(final_sum_kernel, dim3(1), dim3(kRedBlock), 0, st, partials, np, out);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

__device__ inline int64_t qfix(double x) { return static_cast<int64_t>(__builtin_rint(x * kQScale)); }

// fixed-order sum of np block partials by one block (every thread gets it)
__device__ inline double sum_partials(const double* __restrict__ part, int np, double* sh) {
  double s = 0.0;
  for (int t = threadIdx.x; t < np; t += kBlock) s += part[t];
  return block_sum(s, sh);
}

// block 0 of a launch writes the totals of the previous step from its block
// partials (all threads of the block take part)
__device__ inline void write_step_sums(const StepSums& prev) {
  __shared__ double sh[kBlock];
  const double ep = sum_partials(prev.part_e, prev.np, sh);
  __syncthreads();
  const double ek = sum_partials(prev.part_k, prev.np, sh);
  if (threadIdx.x == 0) {
    *prev.e_pot = ep;
    *prev.e_kin = ek;
  }
}

// The kicks v += (dt/2 F) / m and the drift r += dt v are written as explicit
// fused multiply-adds, so that every kernel that applies them rounds alike
// (the same step gives the same bits whichever kernel performs it).

// Outcome of the displacement check of one or more atoms
struct DriftCheck {
  int bad;       // a non-finite or absurd position
  int viol;      // moved by more than half the skin since the last build
  int64_t d2;    // largest |dq|^2 among the atoms below the limit
};

// r += dt v for atom i (``x0``: the position before the drift) and, against
// the fixed-point build snapshot ``qb`` (null: no check), the displacement
// check: |dq| > skin/2 in fixed point (4 |dq|^2 > skin_q^2) is a violation
__device__ inline DriftCheck drift_check(int64_t i, const double* v, const double* x0,
                                         double* __restrict__ pos, double dt, const int64_t* qb,
                                         int64_t skin_q) {
  DriftCheck c{0, 0, 0};
  bool far = false;
  int64_t d2 = 0;
  for (int a = 0; a < 3; ++a) {
    const double x = __fma_rn(dt, v[a], x0[a]);
    pos[3 * i + a] = x;
    if (!isfinite(x) || fabs(x) > 1.0e12) c.bad = 1;
    if (!c.bad && qb) {
      const int64_t dq = qfix(x) - qb[a];
      if (dq > skin_q || dq < -skin_q) far = true;
      else d2 += dq * dq;
    }
  }
  if (qb && (c.bad || far || 4 * d2 > skin_q * skin_q)) c.viol = 1;
  else if (qb) c.d2 = d2;
  return c;
}

__device__ inline DriftCheck merge(DriftCheck a, const DriftCheck& b) {
  a.bad |= b.bad;
  a.viol |= b.viol;
  a.d2 = a.d2 > b.d2 ? a.d2 : b.d2;
  return a;
}

// one set of atomics for the merged checks of several atoms of step
// ``step``: flags[0] bit 3 marks a bad position, flags[1] a violation,
// flags[4] takes the smallest violating step and flags[5] the largest |dq|^2
__device__ inline void record_check(const DriftCheck& c, int64_t* __restrict__ flags, int64_t step) {
  if (c.bad) atomicOr(reinterpret_cast<unsigned long long*>(flags), 8ull);
  if (c.viol) {
    atomicOr(reinterpret_cast<unsigned long long*>(flags + 1), 1ull);
    atomicMin(reinterpret_cast<unsigned long long*>(flags + 4), (unsigned long long)step);
  }
  if (c.d2 > 0) atomicMax(reinterpret_cast<unsigned long long*>(flags + 5), (unsigned long long)c.d2);
}

// v += dt/2 F/m (after v *= *scale when a scale is given) and optionally the
// drift with its displacement check (merged per wave); block 0 first writes
// the totals of ``prev``
__global__ void __launch_bounds__(kBlock) kick_drift_kernel(double* __restrict__ pos, double* __restrict__ vel,
                                                            const double* __restrict__ forces,
                                                            const int32_t* __restrict__ species,
                                                            const double* __restrict__ inv_mass,
                                                            int n_types1, int64_t n, double half_dt,
                                                            double dt,
                                                            int drift, const int64_t* __restrict__ qbuild,
                                                            int64_t skin_q, int64_t* __restrict__ flags,
                                                            StepSums prev, int64_t step,
                                                            const double* __restrict__ scale) {
  if (prev.np > 0 && blockIdx.x == 0) write_step_sums(prev);
  const int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  DriftCheck c{0, 0, 0};
  if (i < n) {
    int a0 = species[i];
    a0 = static_cast<unsigned>(a0) < static_cast<unsigned>(n_types1) ? a0 : n_types1 - 1;
    const double im = inv_mass[a0];
    double v[3];
    for (int a = 0; a < 3; ++a) v[a] = vel[3 * i + a];
    if (scale) {   // the thermostat's velocity scale, applied before the kick
      // (rounded on its own, not contracted into the kick: with s = 1 the kick
      // is then exactly the NVE one)
      const double s = *scale;
      for (int a = 0; a < 3; ++a) v[a] = __dmul_rn(v[a], s);
    }
    for (int a = 0; a < 3; ++a) {
      v[a] = __fma_rn(half_dt * forces[3 * i + a], im, v[a]);
      vel[3 * i + a] = v[a];
    }
    if (drift) {
      const double x0[3] = {pos[3 * i], pos[3 * i + 1], pos[3 * i + 2]};
      int64_t qb[3] = {0, 0, 0};
      if (qbuild)
        for (int a = 0; a < 3; ++a) qb[a] = qbuild[3 * i + a];
      c = drift_check(i, v, x0, pos, dt, qbuild ? qb : nullptr, skin_q);
    }
  }
  if (!drift) return;
  for (int off = 1; off < kWave; off <<= 1) {
    DriftCheck o;
    o.bad = __shfl_xor(c.bad, off);
    o.viol = __shfl_xor(c.viol, off);
    o.d2 = __shfl_xor(c.d2, off);
    c = merge(c, o);
  }
  if ((threadIdx.x & (kWave - 1)) == 0) record_check(c, flags, step);
}

// Force assembly.  The gradient g_e of compact slot c of row b = row_ptr[k]
// sits at the skin position of the edge, grad[b + cskin[b + c]], and the
// gradient of its reverse at the skin position of the reverse,
// grad[skin_rev[b + cskin[b + c]]] (every edge inside r_c has its reverse
// inside r_c, by the exact integer predicate), so a reverse takes one
// gather.  Sixteen lanes per atom, sixteen atoms per group.
//
// With TAIL (a velocity-Verlet step) the lane that holds F_k also applies
// the second half kick v += dt/2 F/m; the group's potential and kinetic
// energies are summed in a fixed order, and each block adds its groups up in
// the order it visits them into partial ``blockIdx.x`` of this step (at most
// kMaxTailBlocks partials, so the step totals are short sums).  One extra
// block writes the totals of the previous step (a separate partial buffer).
// With kick_next the same lane goes on with the first half kick and the
// drift of the next step (drift_check): both use F_k, so the arithmetic is
// that of separate kick kernels.
//
// With VIR the per-centre virial terms W_k of Eq. (forces), formed by the
// backward kernel, are summed the same way into part_v[block][9].
template <bool TAIL, bool VIR>
__global__ void __launch_bounds__(kBlock) forces_kernel(int64_t n, const int64_t* __restrict__ row_ptr,
                                                        const int32_t* __restrict__ ecount,
                                                        const float4* __restrict__ grad,
                                                        const int32_t* __restrict__ cskin,
                                                        const int64_t* __restrict__ skin_rev,
                                                        double* __restrict__ forces, StepTail tl,
                                                        VirialOut vo) {
  constexpr int APG = kBlock / kLanesPerAtom;
  __shared__ double she[APG], shk[APG];
  __shared__ DriftCheck shc[APG];
  __shared__ double shv[VIR ? APG : 1][9];
  // with TAIL the last block only writes the totals of the previous step
  // (off the path of the atoms' blocks)
  const int64_t nblk = TAIL ? gridDim.x - 1 : gridDim.x;
  if (TAIL && blockIdx.x == nblk) {
    if (tl.prev.np > 0) write_step_sums(tl.prev);
    return;
  }
  const int sub = threadIdx.x % kLanesPerAtom, slot = threadIdx.x / kLanesPerAtom;
  const int64_t groups = (n + APG - 1) / APG;
  double blk_e = 0.0, blk_k = 0.0, blk_v = 0.0;   // the block's partials (threads 0, 0..8)
  for (int64_t grp = xcd_block(blockIdx.x, nblk); grp < groups; grp += nblk) {
    const int64_t k = grp * APG + slot;
    // the step's per-atom inputs, requested before the row so that their
    // latency overlaps the gathers
    double im = 0.0, ms = 0.0, eat = 0.0, v0[3] = {0.0, 0.0, 0.0}, x0[3] = {0.0, 0.0, 0.0};
    int64_t qb[3] = {0, 0, 0};
    if (TAIL && sub == 0 && k < n) {
      int a0 = tl.species[k];
      a0 = static_cast<unsigned>(a0) < static_cast<unsigned>(tl.n_types1) ? a0 : tl.n_types1 - 1;
      im = tl.inv_mass[a0];
      ms = tl.mass[a0];
      eat = tl.e_atom[k];
      for (int a = 0; a < 3; ++a) v0[a] = tl.vel[3 * k + a];
      if (tl.kick_next) {
        for (int a = 0; a < 3; ++a) x0[a] = tl.pos[3 * k + a];
        if (tl.qbuild)
          for (int a = 0; a < 3; ++a) qb[a] = tl.qbuild[3 * k + a];
      }
    }
    double fx = 0.0, fy = 0.0, fz = 0.0;
    double w[VIR ? 9 : 1];   // the centre's virial term, on the lane that sums it
    for (int c = 0; c < (VIR ? 9 : 1); ++c) w[c] = 0.0;
    if (VIR && sub == 0 && k < n)
      for (int c = 0; c < 9; ++c) w[c] = vo.atom[9 * k + c];
    if (k < n) {
      const int64_t b = row_ptr[k], e = b + ecount[k];
      for (int64_t c = b + sub; c < e; c += kLanesPerAtom) {
        const int64_t s = b + cskin[c];
        const float4 g = grad[s];
        const int64_t sr = skin_rev[s];
        const float4 r = sr >= 0 ? grad[sr] : g;   // a valid list always has the reverse
        fx += double(g.x) - double(r.x);
        fy += double(g.y) - double(r.y);
        fz += double(g.z) - double(r.z);
      }
    }
    for (int off = 1; off < kLanesPerAtom; off <<= 1) {
      fx += __shfl_xor(fx, off, kLanesPerAtom);
      fy += __shfl_xor(fy, off, kLanesPerAtom);
      fz += __shfl_xor(fz, off, kLanesPerAtom);
    }
    double ep = 0.0, ek = 0.0;
    DriftCheck chk{0, 0, 0};
    if (sub == 0 && k < n) {
      forces[3 * k] = fx;
      forces[3 * k + 1] = fy;
      forces[3 * k + 2] = fz;
      if (TAIL) {
        const double f[3] = {fx, fy, fz};
        double v[3], v2 = 0.0;
        for (int a = 0; a < 3; ++a) {
          v[a] = __fma_rn(tl.half_dt * f[a], im, v0[a]);
          v2 += v[a] * v[a];
        }
        // 1 u (A/fs)^2 = 103.6427 eV (CODATA 2018 atomic mass unit and elementary charge)
        ek = 0.5 * ms * v2 * (1.66053906660e-17 / 1.602176634e-19);
        ep = eat;
        if (tl.kick_next) {
          for (int a = 0; a < 3; ++a) v[a] = __fma_rn(tl.half_dt * f[a], im, v[a]);
          chk = drift_check(k, v, x0, tl.pos, tl.dt, tl.qbuild ? qb : nullptr, tl.skin_q);
        }
        for (int a = 0; a < 3; ++a) tl.vel[3 * k + a] = v[a];
      }
    }
    if (TAIL || VIR) {
      if (sub == 0) {
        if (TAIL) {
          she[slot] = ep;
          shk[slot] = ek;
          shc[slot] = chk;
        }
        if (VIR)
          for (int c = 0; c < 9; ++c) shv[slot][c] = k < n ? w[c] : 0.0;
      }
      __syncthreads();
      if (TAIL && threadIdx.x == 0) {
        double se = she[0], sk = shk[0];
        DriftCheck c = shc[0];
        for (int q = 1; q < APG; ++q) {
          se += she[q];
          sk += shk[q];
          c = merge(c, shc[q]);
        }
        blk_e += se;
        blk_k += sk;
        if (tl.kick_next) record_check(c, tl.flags, tl.next_step);
      }
      if (VIR && threadIdx.x < 9) {
        const int c = threadIdx.x;
        double sv = shv[0][c];
        for (int q = 1; q < APG; ++q) sv += shv[q][c];
        blk_v += sv;
      }
      __syncthreads();
    }
  }
  // one partial per block: its groups in the order it visited them
  if (TAIL && threadIdx.x == 0) {
    tl.part_e[blockIdx.x] = blk_e;
    tl.part_k[blockIdx.x] = blk_k;
  }
  if (VIR && threadIdx.x < 9) vo.part_v[9 * blockIdx.x + threadIdx.x] = blk_v;
}

// ---- Nose-Hoover chain (NVT) ------------------------------------------------
// The chain of Martyna, Klein and Tuckerman (J. Chem. Phys. 97, 2635, 1992)
// with masses Q_1 = N_f kT tau^2, Q_k = kT tau^2, propagated over dt/2 by the
// Trotter factorisation of Martyna, Tuckerman, Tobias and Klein (Mol. Phys.
// 87, 1117, 1996), one pass: thermostat velocities from the end of the chain
// inwards, the particle velocities scaled by exp(-dt/2 v_1), the positions
// xi_k advanced by dt/2 v_k, and the velocities outwards again.  Chain forces:
// G_1 = (2K - N_f kT)/Q_1, G_k = (Q_{k-1} v_{k-1}^2 - kT)/Q_k.  Returns the
// velocity scale; ``ke`` is the kinetic energy before the scaling.
__device__ double chain_half_step(const NhcArgs& a, double* xi, double* v, double ke) {
  const int M = a.M;
  const double q = 0.25 * a.dt, e = 0.125 * a.dt;
  auto force = [&](int k, double kin) {
    return k == 0 ? (2.0 * kin - a.nf * a.kT) / a.Q[0]
                  : (a.Q[k - 1] * v[k - 1] * v[k - 1] - a.kT) / a.Q[k];
  };
  auto update = [&](int k, double kin) {
    if (k == M - 1) {
      v[k] += q * force(k, kin);
    } else {
      const double f = exp(-e * v[k + 1]);
      v[k] = (v[k] * f + q * force(k, kin)) * f;
    }
  };
  for (int k = M - 1; k >= 0; --k) update(k, ke);
  const double s = exp(-0.5 * a.dt * v[0]);
  ke *= s * s;
  for (int k = 0; k < M; ++k) xi[k] += 0.5 * a.dt * v[k];
  for (int k = 0; k < M; ++k) update(k, ke);
  return s;
}

// fixed-order sum over p < np of part[stride p + c] by one block
__device__ inline double sum_strided(const double* __restrict__ part, int64_t np, int stride, int c,
                                     double* sh) {
  double s = 0.0;
  for (int64_t p = threadIdx.x; p < np; p += kBlock) s += part[stride * p + c];
  return block_sum(s, sh);
}

// One block.  Closing a step: its kinetic energy K (partials part_k), the
// chain half step, K s^2 as the step's kinetic energy, the potential energy,
// the thermostat energy and the virial of the step.  Opening a step: the
// chain half step for the current K.  state[2M] = the product of the scales
// of both, which the next kick (or launch_scale) applies.
__global__ void __launch_bounds__(kBlock) nhc_kernel(NhcArgs a) {
  __shared__ double sh[kBlock];
  double ke = sum_strided(a.part_k, a.np, 1, 0, sh);
  __syncthreads();
  double pe = 0.0, vir[9];
  if (a.close_prev && a.e_pot) {
    pe = sum_strided(a.part_e, a.np, 1, 0, sh);
    __syncthreads();
  }
  for (int c = 0; c < 9; ++c) {
    vir[c] = 0.0;
    if (a.close_prev && a.virial) {
      vir[c] = sum_strided(a.part_v, a.np, 9, c, sh);
      __syncthreads();
    }
  }
  if (threadIdx.x != 0) return;
  double* xi = a.state;
  double* v = a.state + a.M;
  double scale = 1.0;
  if (a.close_prev) {
    const double s = chain_half_step(a, xi, v, ke);
    ke *= s * s;
    scale *= s;
    double eth = a.nf * a.kT * xi[0];
    for (int k = 0; k < a.M; ++k) eth += 0.5 * a.Q[k] * v[k] * v[k] + (k > 0 ? a.kT * xi[k] : 0.0);
    if (a.e_pot) *a.e_pot = pe;
    if (a.e_kin) *a.e_kin = ke;
    if (a.e_thermo) *a.e_thermo = eth;
    if (a.virial)
      for (int c = 0; c < 9; ++c) a.virial[c] = vir[c];
  }
  if (a.open_next) scale *= chain_half_step(a, xi, v, ke);
  a.state[2 * a.M] = scale;
}

// block partials (256 atoms each, fixed tree) of the kinetic energy
__global__ void __launch_bounds__(kBlock) kinetic_kernel(const double* __restrict__ vel,
                                                         const int32_t* __restrict__ species,
                                                         const double* __restrict__ mass,
                                                         int n_types1, int64_t n,
                                                         double* __restrict__ part_k) {
  __shared__ double sh[kBlock];
  const int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  double ek = 0.0;
  if (i < n) {
    int a0 = species[i];
    a0 = static_cast<unsigned>(a0) < static_cast<unsigned>(n_types1) ? a0 : n_types1 - 1;
    double v2 = 0.0;
    for (int a = 0; a < 3; ++a) v2 += vel[3 * i + a] * vel[3 * i + a];
    ek = 0.5 * mass[a0] * v2 * (1.66053906660e-17 / 1.602176634e-19);
  }
  const double tk = block_sum(ek, sh);
  if (threadIdx.x == 0) part_k[blockIdx.x] = tk;
}

__global__ void __launch_bounds__(kBlock) scale_kernel(double* __restrict__ vel, int64_t n3,
                                                       const double* __restrict__ scale) {
  const int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i < n3) vel[i] = vel[i] * *scale;
}

__global__ void __launch_bounds__(kBlock) final_step_kernel(StepSums prev) {
  __shared__ double sh[kBlock];
  const double ep = sum_partials(prev.part_e, prev.np, sh);
  __syncthreads();
  const double ek = sum_partials(prev.part_k, prev.np, sh);
  if (threadIdx.x == 0) {
    *prev.e_pot = ep;
    *prev.e_kin = ek;
  }
}

__global__ void __launch_bounds__(kBlock) snapshot_kernel(const double* __restrict__ pos, int64_t n,
                                                          int64_t* __restrict__ qbuild) {
  int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i >= 3 * n) return;
  qbuild[i] = qfix(pos[i]);
}

__global__ void set_flag_kernel(int64_t* flags, int idx, int64_t value) {
  if (threadIdx.x == 0) flags[idx] = value;
}

__global__ void __launch_bounds__(kBlock) zero_i64_kernel(int64_t* __restrict__ p, int64_t n) {
  for (int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kBlock)
    p[i] = 0;
}

int blocks_for(int64_t n) {
  int64_t b = (n + kBlock - 1) / kBlock;
  return static_cast<int>(b < 1 ? 1 : b);
}

}  // namespace

int launch_forces(int64_t n, const int64_t* row_ptr, const int32_t* ecount, const float4* grad,
                  const int32_t* cskin, const int64_t* skin_rev,
                  double* forces, const StepTail* tail, const VirialOut* vir, hipStream_t st) {
  const int64_t blocks = tail_partial_count(n);
  const StepTail tl = tail ? *tail : StepTail{};
  const VirialOut vo = vir ? *vir : VirialOut{};
  if (vir && (!vir->part_v || !vir->atom)) return DPA4C_ERR_INVALID_ARG;
  const dim3 grid(static_cast<unsigned>(blocks + (tail ? 1 : 0)));
  if (tail && vir)
    hipLaunchKernelGGL((forces_kernel<true, true>), grid, dim3(kBlock), 0, st, n, row_ptr, ecount,
                       grad, cskin, skin_rev, forces, tl, vo);
  else if (tail)
    hipLaunchKernelGGL((forces_kernel<true, false>), grid, dim3(kBlock), 0, st, n, row_ptr, ecount,
                       grad, cskin, skin_rev, forces, tl, vo);
  else if (vir)
    hipLaunchKernelGGL((forces_kernel<false, true>), grid, dim3(kBlock), 0, st, n, row_ptr, ecount,
                       grad, cskin, skin_rev, forces, tl, vo);
  else
    hipLaunchKernelGGL((forces_kernel<false, false>), grid, dim3(kBlock), 0, st, n, row_ptr,
                       ecount, grad, cskin, skin_rev, forces, tl, vo);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

// out[c] = sum over p < np of part[ncomp p + c], c < ncomp, in a fixed order
// (one block)
__global__ void __launch_bounds__(kRedBlock) sum_components_kernel(const double* __restrict__ part,
                                                                   int64_t np, int ncomp,
                                                                   double* __restrict__ out) {
  __shared__ double sh[kRedBlock];
  for (int c = 0; c < ncomp; ++c) {
    double s = 0.0;
    for (int64_t p = threadIdx.x; p < np; p += kRedBlock) s += part[ncomp * p + c];
    const double tot = block_sum(s, sh);
    if (threadIdx.x == 0) out[c] = tot;
    __syncthreads();
  }
}

int launch_sum_components(const double* part, int64_t np, int ncomp, double* out, hipStream_t st) {
  hipLaunchKernelGGL(sum_components_kernel, dim3(1), dim3(kRedBlock), 0, st, part, np, ncomp, out);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_energy(int64_t n, const double* e_atom, double* partials, double* out, hipStream_t st) {
  return fixed_sum(e_atom, n, partials, out, st);
}

int launch_kick_drift(double* pos, double* vel, const double* forces, const int32_t* species,
                      const double* inv_mass, int n_types1, int64_t n, double dt, int drift,
                      const int64_t* qbuild, int64_t skin_q, int64_t* flags, StepSums prev,
                      int64_t step, const double* scale, hipStream_t st) {
  hipLaunchKernelGGL(kick_drift_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, st, pos, vel, forces,
                     species, inv_mass, n_types1, n, 0.5 * dt, dt, drift, qbuild, skin_q, flags,
                     prev, step, scale);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_nhc(const NhcArgs& a, hipStream_t st) {
  if (a.M < 1 || a.M > kMaxChain || !a.state || !a.part_k || a.np < 1) return DPA4C_ERR_INVALID_ARG;
  hipLaunchKernelGGL(nhc_kernel, dim3(1), dim3(kBlock), 0, st, a);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int kinetic_partial_count(int64_t n) { return blocks_for(n); }

int launch_kinetic(const double* vel, const int32_t* species, const double* mass, int n_types1,
                   int64_t n, double* part_k, hipStream_t st) {
  hipLaunchKernelGGL(kinetic_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, st, vel, species, mass,
                     n_types1, n, part_k);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_scale(double* vel, int64_t n, const double* scale, hipStream_t st) {
  hipLaunchKernelGGL(scale_kernel, dim3(blocks_for(3 * n)), dim3(kBlock), 0, st, vel, 3 * n, scale);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_final_step(StepSums prev, hipStream_t st) {
  if (prev.np <= 0) return 0;
  hipLaunchKernelGGL(final_step_kernel, dim3(1), dim3(kBlock), 0, st, prev);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

// blocks of the force assembly, one energy (and virial) partial each
int tail_partial_count(int64_t n) {
  const int64_t g = (n + kBlock / kLanesPerAtom - 1) / (kBlock / kLanesPerAtom);
  return static_cast<int>(g < 1 ? 1 : (g > kMaxTailBlocks ? kMaxTailBlocks : g));
}

int launch_snapshot_q(const double* pos, int64_t n, int64_t* qbuild, hipStream_t st) {
  hipLaunchKernelGGL(snapshot_kernel, dim3(blocks_for(3 * n)), dim3(kBlock), 0, st, pos, n, qbuild);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_set_flag(int64_t* flags, int idx, int64_t value, hipStream_t st) {
  hipLaunchKernelGGL(set_flag_kernel, dim3(1), dim3(64), 0, st, flags, idx, value);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_zero_i64(int64_t* p, int64_t n, hipStream_t st) {
  if (n <= 0) return 0;
  int b = blocks_for(n);
  hipLaunchKernelGGL(zero_i64_kernel, dim3(b < 1024 ? b : 1024), dim3(kBlock), 0, st, p, n);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int partial_count(int64_t n) {
  int64_t np = (n + kRedBlock * kRedPer - 1) / (kRedBlock * kRedPer);
  return static_cast<int>(np < 1 ? 1 : np);
}

}  // namespace dpa4c
