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

// The reverse of compact slot s is cidx[skin_rev[sidx[s]]]: the compact slot
// of the reverse skin edge (every edge inside r_c has its reverse inside r_c).
__global__ void __launch_bounds__(kBlock) forces_kernel(int64_t n, const int64_t* __restrict__ row_ptr,
                                                        const int32_t* __restrict__ ecount,
                                                        const float4* __restrict__ grad,
                                                        const int32_t* __restrict__ sidx,
                                                        const int32_t* __restrict__ skin_rev,
                                                        const int32_t* __restrict__ cidx,
                                                        double* __restrict__ forces) {
  const int sub = threadIdx.x % kLanesPerAtom;
  const int64_t per_grid = int64_t(gridDim.x) * (kBlock / kLanesPerAtom);
  for (int64_t k = blockIdx.x * int64_t(kBlock / kLanesPerAtom) + threadIdx.x / kLanesPerAtom; k < n;
       k += per_grid) {
    const int64_t b = row_ptr[k], e = b + ecount[k];
    double fx = 0.0, fy = 0.0, fz = 0.0;
    for (int64_t s = b + sub; s < e; s += kLanesPerAtom) {
      const float4 g = grad[s];
      const int32_t sr = skin_rev[sidx[s]];
      const int32_t c = sr >= 0 ? cidx[sr] : -1;
      const float4 r = c >= 0 ? grad[c] : g;   // a valid list always has the reverse
      fx += double(g.x) - double(r.x);
      fy += double(g.y) - double(r.y);
      fz += double(g.z) - double(r.z);
    }
    for (int off = 1; off < kLanesPerAtom; off <<= 1) {
      fx += __shfl_xor(fx, off, kLanesPerAtom);
      fy += __shfl_xor(fy, off, kLanesPerAtom);
      fz += __shfl_xor(fz, off, kLanesPerAtom);
    }
    if (sub == 0) {
      forces[3 * k] = fx;
      forces[3 * k + 1] = fy;
      forces[3 * k + 2] = fz;
    }
  }
}

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

// v += dt/2 F/m; optionally r += dt v and, against the fixed-point positions
// of the last build, flag a rebuild when some atom moved by more than half
// the skin (4 |dq|^2 > skin_q^2): flags[1] is set, flags[4] takes the
// smallest such step index and flags[5] the largest |dq|^2 below the limit.
// fixed-order sum of np block partials by one block (every thread gets it)
__device__ inline double sum_partials(const double* __restrict__ part, int np, double* sh) {
  double s = 0.0;
  for (int t = threadIdx.x; t < np; t += kBlock) s += part[t];
  return block_sum(s, sh);
}

__global__ void __launch_bounds__(kBlock) kick_drift_kernel(double* __restrict__ pos, double* __restrict__ vel,
                                                            const double* __restrict__ forces,
                                                            const int32_t* __restrict__ species,
                                                            const double* __restrict__ inv_mass,
                                                            int n_types1, int64_t n, double half_dt,
                                                            double dt,
                                                            int drift, const int64_t* __restrict__ qbuild,
                                                            int64_t skin_q, int64_t* __restrict__ flags,
                                                            StepSums prev, int64_t step) {
  if (prev.np > 0 && blockIdx.x == 0) {
    // totals of the previous step from the block partials of its tail kernel
    __shared__ double sh[kBlock];
    const double ep = sum_partials(prev.part_e, prev.np, sh);
    __syncthreads();
    const double ek = sum_partials(prev.part_k, prev.np, sh);
    if (threadIdx.x == 0) {
      *prev.e_pot = ep;
      *prev.e_kin = ek;
    }
  }
  int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  if (i >= n) return;
  int a0 = species[i];
  a0 = static_cast<unsigned>(a0) < static_cast<unsigned>(n_types1) ? a0 : n_types1 - 1;
  const double im = inv_mass[a0];
  double v[3], x[3];
  for (int a = 0; a < 3; ++a) {
    v[a] = vel[3 * i + a] + half_dt * forces[3 * i + a] * im;
    vel[3 * i + a] = v[a];
  }
  if (!drift) return;
  bool bad = false;
  int64_t d2 = 0;
  bool far = false;
  for (int a = 0; a < 3; ++a) {
    x[a] = pos[3 * i + a] + dt * v[a];
    pos[3 * i + a] = x[a];
    if (!isfinite(x[a]) || fabs(x[a]) > 1.0e12) bad = true;
    if (!bad && qbuild) {
      int64_t dq = qfix(x[a]) - qbuild[3 * i + a];
      if (dq > skin_q || dq < -skin_q) far = true;
      else d2 += dq * dq;
    }
  }
  if (bad) atomicOr(reinterpret_cast<unsigned long long*>(flags), 8ull);
  if (!qbuild) return;
  if (bad || far || 4 * d2 > skin_q * skin_q) {
    atomicOr(reinterpret_cast<unsigned long long*>(flags + 1), 1ull);
    atomicMin(reinterpret_cast<unsigned long long*>(flags + 4), (unsigned long long)step);
  } else {
    atomicMax(reinterpret_cast<unsigned long long*>(flags + 5), (unsigned long long)d2);
  }
}

// Second half kick v += dt/2 F/m, then the block partials (fixed tree) of
// the potential energy sum_i E_i and of the kinetic energy of the block's
// atoms; the next kick_drift_kernel (or final_step_kernel) adds the partials.
__global__ void __launch_bounds__(kBlock) tail_kernel(int64_t n, double* __restrict__ vel,
                                                      const double* __restrict__ forces,
                                                      const int32_t* __restrict__ species,
                                                      const double* __restrict__ inv_mass,
                                                      const double* __restrict__ mass,
                                                      int n_types1, double half_dt,
                                                      const double* __restrict__ e_atom,
                                                      double* __restrict__ part_e,
                                                      double* __restrict__ part_k) {
  __shared__ double sh[kBlock];
  const int64_t i = blockIdx.x * int64_t(kBlock) + threadIdx.x;
  double ek = 0.0, ep = 0.0;
  if (i < n) {
    int a0 = species[i];
    a0 = static_cast<unsigned>(a0) < static_cast<unsigned>(n_types1) ? a0 : n_types1 - 1;
    const double im = inv_mass[a0];
    double v2 = 0.0;
    for (int a = 0; a < 3; ++a) {
      const double v = vel[3 * i + a] + half_dt * forces[3 * i + a] * im;
      vel[3 * i + a] = v;
      v2 += v * v;
    }
    // 1 u (A/fs)^2 = 103.6427 eV (CODATA 2018 atomic mass unit and elementary charge)
    ek = 0.5 * mass[a0] * v2 * (1.66053906660e-17 / 1.602176634e-19);
    ep = e_atom[i];
  }
  const double te = block_sum(ep, sh);
  __syncthreads();
  const double tk = block_sum(ek, sh);
  if (threadIdx.x == 0) {
    part_e[blockIdx.x] = te;
    part_k[blockIdx.x] = tk;
  }
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

int blocks_for(int64_t n) {
  int64_t b = (n + kBlock - 1) / kBlock;
  return static_cast<int>(b < 1 ? 1 : b);
}

}  // namespace

int launch_forces(int64_t n, const int64_t* row_ptr, const int32_t* ecount, const float4* grad,
                  const int32_t* sidx, const int32_t* skin_rev, const int32_t* cidx,
                  double* forces, hipStream_t st) {
  int64_t blocks = (n + (kBlock / kLanesPerAtom) - 1) / (kBlock / kLanesPerAtom);
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(forces_kernel, dim3(blocks), dim3(kBlock), 0, st, n, row_ptr, ecount, grad,
                     sidx, skin_rev, cidx, forces);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_energy(int64_t n, const double* e_atom, double* partials, double* out, hipStream_t st) {
  return fixed_sum(e_atom, n, partials, out, st);
}

int launch_kick_drift(double* pos, double* vel, const double* forces, const int32_t* species,
                      const double* inv_mass, int n_types1, int64_t n, double dt, int drift,
                      const int64_t* qbuild, int64_t skin_q, int64_t* flags, StepSums prev,
                      int64_t step, hipStream_t st) {
  hipLaunchKernelGGL(kick_drift_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, st, pos, vel, forces,
                     species, inv_mass, n_types1, n, 0.5 * dt, dt, drift, qbuild, skin_q, flags,
                     prev, step);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_tail(int64_t n, double* vel, const double* forces, const int32_t* species,
                const double* inv_mass, const double* mass, int n_types1, double dt,
                const double* e_atom, double* part_e, double* part_k, hipStream_t st) {
  hipLaunchKernelGGL(tail_kernel, dim3(blocks_for(n)), dim3(kBlock), 0, st, n, vel, forces,
                     species, inv_mass, mass, n_types1, 0.5 * dt, e_atom, part_e, part_k);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int launch_final_step(StepSums prev, hipStream_t st) {
  if (prev.np <= 0) return 0;
  hipLaunchKernelGGL(final_step_kernel, dim3(1), dim3(kBlock), 0, st, prev);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

int tail_partial_count(int64_t n) { return blocks_for(n); }

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

int partial_count(int64_t n) {
  int64_t np = (n + kRedBlock * kRedPer - 1) / (kRedBlock * kRedPer);
  return static_cast<int>(np < 1 ? 1 : np);
}

}  // namespace dpa4c
