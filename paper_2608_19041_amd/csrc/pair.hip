// Ordered type-pair cache, Eq. (pairfilm): evaluated once per ordered pair
// (a, b) of the type table (including the padding type), in float64, and
// stored float32 in the lane layout of the edge kernels:
//   pair[(a*(T+1) + b)][j][k][PW],  channel c = k + LPE*j,
//   entries (gamma_c, beta_c, U_c0 .. U_c,R-1).
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "launch.h"

namespace dpa4c {

__global__ void __launch_bounds__(256) pair_cache_kernel(const float* __restrict__ type_embed,
                                                         const float* __restrict__ wp_in,
                                                         const float* __restrict__ wp_out,
                                                         int C0, int Hp, int R, int T1, int LPE,
                                                         float* __restrict__ out) {
  extern __shared__ double sh[];
  double* z = sh;              // [2 C0]
  double* hid = sh + 2 * C0;   // [Hp]
  const int pair = blockIdx.x;
  const int a = pair / T1, b = pair % T1;
  for (int t = threadIdx.x; t < 2 * C0; t += blockDim.x)
    z[t] = t < C0 ? type_embed[a * C0 + t] : type_embed[b * C0 + (t - C0)];
  __syncthreads();
  for (int k = threadIdx.x; k < Hp; k += blockDim.x) {
    double g = 0.0, v = 0.0;
    for (int n = 0; n < 2 * C0; ++n) {
      g += z[n] * (double)wp_in[n * 2 * Hp + k];
      v += z[n] * (double)wp_in[n * 2 * Hp + Hp + k];
    }
    hid[k] = g / (1.0 + exp(-g)) * v;       // SwiGLU, Eq. (swiglu)
  }
  __syncthreads();
  const int PW = 2 + R;
  const int width = C0 * PW;
  for (int o = threadIdx.x; o < width; o += blockDim.x) {
    double p = 0.0;
    for (int k = 0; k < Hp; ++k) p += hid[k] * (double)wp_out[k * width + o];
    p *= 0.1;
    int c, slot;
    double val;
    if (o < C0) {
      c = o; slot = 0; val = 1.0 + tanh(p);                         // gamma
    } else if (o < 2 * C0) {
      c = o - C0; slot = 1; val = z[c] + z[C0 + c] + tanh(p);       // beta
    } else {
      c = (o - 2 * C0) / R; slot = 2 + (o - 2 * C0) % R; val = tanh(p);  // U
    }
    int k = c % LPE, j = c / LPE;
    out[((size_t(pair) * (C0 / LPE) + j) * LPE + k) * PW + slot] = static_cast<float>(val);
  }
}

int launch_pair_cache(dpa4c_model* m, const float* wp_in, const float* wp_out) {
  const int T1 = m->n_types + 1;
  size_t shmem = sizeof(double) * (2 * m->C0 + m->Hp);
  hipLaunchKernelGGL(pair_cache_kernel, dim3(T1 * T1), dim3(256), shmem, 0, m->type_embed,
                     wp_in, wp_out, m->C0, m->Hp, m->R, T1, m->C[1], m->pair);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace dpa4c
