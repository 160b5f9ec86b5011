// Plain fp32 GEMM on the matrix cores (v_mfma_f32_16x16x4_f32) with an
// optional fused epilogue (bias + SiLU + residual, or residual + product).
// The energy path uses the per-atom kernel; this one backs the exported
// dpa4c_debug_gemm entry used to check the MFMA operand layout.
#include <hip/hip_runtime.h>

#include "../../include/dpa4c.h"
#include "launch.h"

namespace dpa4c {

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int BM = 64, BN = 64, BK = 16;
constexpr int kThreads = 256;

__device__ inline float sigmoidf(float z) { return 1.0f / (1.0f + __expf(-z)); }

struct Epilogue {
  int mode;                 // 0: forward activation, 1: backward product
  const float* bias;        // [N]           (mode 0)
  const float* res_vec;     // [N] or null   (mode 1)
  const float* res_mat;     // [M][ldr] or null (mode 0 and 1)
  int ldr;
  float* aux;               // mode 0: SiLU'(pre) [M][ldc]
  const float* mul;         // mode 1: multiply after the residual, [M][ldc], or null
  float* out_h;             // mode 1: store of the value before ``mul`` or null
};

// C[M][N] (row stride ldc) = A[M][K] (stride lda) * B[K][N] (stride ldb) + epilogue.
// K is a multiple of BK; M and N are bounds-checked.
__global__ void __launch_bounds__(kThreads) gemm_kernel(const float* __restrict__ A, int lda,
                                                        const float* __restrict__ B, int ldb,
                                                        float* C, int ldc, int M, int N, int K,
                                                        Epilogue ep) {
  __shared__ float As[BM][BK + 1];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int row0 = blockIdx.y * BM, col0 = blockIdx.x * BN;
  v4f acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = v4f{0.f, 0.f, 0.f, 0.f};

  // loader coordinates
  const int ar = tid >> 2, ak = (tid & 3) * 4;       // A: 64 rows x 16 k
  const int bk = tid >> 4, bn = (tid & 15) * 4;      // B: 16 k x 64 cols
  for (int k0 = 0; k0 < K; k0 += BK) {
    {
      int r = row0 + ar;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (r < M) v = *reinterpret_cast<const float4*>(A + size_t(r) * lda + k0 + ak);
      As[ar][ak + 0] = v.x;
      As[ar][ak + 1] = v.y;
      As[ar][ak + 2] = v.z;
      As[ar][ak + 3] = v.w;
    }
    {
      int c = col0 + bn;
      const float* src = B + size_t(k0 + bk) * ldb + c;
      float4 v;
      if (c + 3 < N) {
        v = *reinterpret_cast<const float4*>(src);
      } else {
        v.x = c + 0 < N ? src[0] : 0.f;
        v.y = c + 1 < N ? src[1] : 0.f;
        v.z = c + 2 < N ? src[2] : 0.f;
        v.w = c + 3 < N ? src[3] : 0.f;
      }
      *reinterpret_cast<float4*>(&Bs[bk][bn]) = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      const int kr = kk + (lane >> 4);
      float a0 = As[wm * 32 + (lane & 15)][kr];
      float a1 = As[wm * 32 + 16 + (lane & 15)][kr];
      float b0 = Bs[kr][wn * 32 + (lane & 15)];
      float b1 = Bs[kr][wn * 32 + 16 + (lane & 15)];
      acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    __syncthreads();
  }
  // epilogue: tile (ti, tj), register r -> row 4*(lane/16) + r, column lane%16
#pragma unroll
  for (int ti = 0; ti < 2; ++ti)
#pragma unroll
    for (int tj = 0; tj < 2; ++tj)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + wm * 32 + ti * 16 + 4 * (lane >> 4) + r;
        const int col = col0 + wn * 32 + tj * 16 + (lane & 15);
        if (row >= M || col >= N) continue;
        float v = acc[ti][tj][r];
        const size_t o = size_t(row) * ldc + col;
        if (ep.mode == 0) {
          float pre = v + (ep.bias ? ep.bias[col] : 0.0f);
          float sg = sigmoidf(pre);
          float h = pre * sg;
          if (ep.res_mat) h += ep.res_mat[size_t(row) * ep.ldr + col];
          C[o] = h;
          if (ep.aux) ep.aux[o] = sg * (1.0f + pre * (1.0f - sg));
        } else {
          if (ep.res_vec) v += ep.res_vec[col];
          if (ep.res_mat) v += ep.res_mat[size_t(row) * ep.ldr + col];
          if (ep.out_h) ep.out_h[o] = v;
          if (ep.mul) v *= ep.mul[o];
          C[o] = v;
        }
      }
}

int gemm(const float* A, int lda, const float* B, int ldb, float* C, int ldc, int M, int N, int K,
         const Epilogue& ep, hipStream_t st) {
  if (K % BK || lda % 4 || ldb % 4 || M < 0) {
    set_error("gemm: K and leading dimensions must be multiples of 16 / 4");
    return DPA4C_ERR_INVALID_ARG;
  }
  if (M == 0) return 0;
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  hipLaunchKernelGGL(gemm_kernel, grid, dim3(kThreads), 0, st, A, lda, B, ldb, C, ldc, M, N, K, ep);
  DPA4C_HIP_TRY(hipGetLastError());
  return 0;
}

}  // namespace

int launch_gemm_test(const float* A, const float* B, float* C, int M, int N, int K,
                     hipStream_t st) {
  Epilogue ep{};
  ep.mode = 1;
  return gemm(A, K, B, N, C, N, M, N, K, ep, st);
}

}  // namespace dpa4c
