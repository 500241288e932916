// Matrix products C = A W^T for the rollout: activations A [rows, K] times
// weights W [N, K] (both K-contiguous), fp32 results, optional split over K.
//
// bf16: gfx950 MFMA v_mfma_f32_16x16x32_bf16.  A wave owns 16 output columns
// and WM tiles of 16 rows; every lane streams 16-byte slices of its weight row
// straight from HBM (the weights are read once per row block), and the A
// fragments come from L2 (activations are small next to weights).  The
// activation arrives as hi/lo bf16 planes; each fragment takes two MFMAs
// (W*hi, W*lo) into the same fp32 accumulator.  Operand
// lane layout of the 16x16x32 MFMA: lane l supplies row (l % 16), k-slice
// 8*(l / 16) .. +7 of A and column (l % 16), the same k-slice of B; it
// receives C rows 4*(l / 16) .. +3 of column (l % 16).
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

constexpr int GEMM_WM = 4;              // 4 x 16 = 64 rows per block
constexpr int GEMM_WAVES = 4;           // 4 x 16 = 64 columns per block

__device__ __forceinline__ bf16x8_t load_bf16x8(const bf16_t* p) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  return __builtin_bit_cast(bf16x8_t, u);
}

__global__ __launch_bounds__(256) void k_gemm_bf16(const bf16_t* __restrict__ A, int lda, int64_t a_plane,
                                                   const bf16_t* __restrict__ W, int ldw,
                                                   float* __restrict__ C, int ldc, int64_t split_stride,
                                                   const int* __restrict__ d_rows, int N, int K,
                                                   int k_per_split) {
  const int M = *d_rows;
  const int row0 = blockIdx.y * (16 * GEMM_WM);
  if (row0 >= M) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = (blockIdx.x * GEMM_WAVES + wave) * 16;
  if (n0 >= N) return;
  const int kb = blockIdx.z * k_per_split;
  const int ke = min(K, kb + k_per_split);
  const int lr = lane & 15, lk = (lane >> 4) * 8;

  const bf16_t* wp = W + (int64_t)(n0 + lr) * ldw + lk;
  const bf16_t* ap[GEMM_WM];
#pragma unroll
  for (int i = 0; i < GEMM_WM; ++i) {
    int r = min(row0 + i * 16 + lr, M - 1);   // clamp: rows past M are computed, never stored
    ap[i] = A + (int64_t)r * lda + lk;
  }
  f32x4_t acc[GEMM_WM];
#pragma unroll
  for (int i = 0; i < GEMM_WM; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll 2
  for (int k = kb; k < ke; k += 32) {
    bf16x8_t b = load_bf16x8(wp + k);
#pragma unroll
    for (int i = 0; i < GEMM_WM; ++i) {
      bf16x8_t ah = load_bf16x8(ap[i] + k);
      bf16x8_t al = load_bf16x8(ap[i] + a_plane + k);
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b, acc[i], 0, 0, 0);
      acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b, acc[i], 0, 0, 0);
    }
  }
  float* cp = C + blockIdx.z * split_stride;
  const int col = n0 + lr;
#pragma unroll
  for (int i = 0; i < GEMM_WM; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int r = row0 + i * 16 + (lane >> 4) * 4 + j;
      if (r < M) cp[(int64_t)r * ldc + col] = acc[i][j];
    }
  }
}

// fp32 models: plain fp32 FMA, one thread per output, 64 columns x 4 rows per block.
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const float* __restrict__ W, int ldw,
                                                  float* __restrict__ C, int ldc, int64_t split_stride,
                                                  const int* __restrict__ d_rows, int N, int K,
                                                  int k_per_split) {
  const int M = *d_rows;
  const int r = blockIdx.y * 4 + (threadIdx.x >> 6);
  const int n = blockIdx.x * 64 + (threadIdx.x & 63);
  if (r >= M || n >= N) return;
  const int kb = blockIdx.z * k_per_split;
  const int ke = min(K, kb + k_per_split);
  const float* a = A + (int64_t)r * lda;
  const float* w = W + (int64_t)n * ldw;
  float acc = 0.f;
  for (int k = kb; k < ke; ++k) acc = fmaf(a[k], w[k], acc);
  C[blockIdx.z * split_stride + (int64_t)r * ldc + n] = acc;
}

}  // namespace

hipError_t launch_gemm(int dtype, const void* A, int lda, int64_t a_plane, const void* W, int ldw, float* C, int ldc,
                       int64_t split_stride, const int* d_rows, int rows_ub, int N, int K, int splits,
                       int k_per_split, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (dtype == 1) {
    dim3 grid((N + 16 * GEMM_WAVES - 1) / (16 * GEMM_WAVES), (rows_ub + 16 * GEMM_WM - 1) / (16 * GEMM_WM), splits);
    hipLaunchKernelGGL(k_gemm_bf16, grid, dim3(256), 0, st, (const bf16_t*)A, lda, a_plane, (const bf16_t*)W, ldw, C,
                       ldc, split_stride, d_rows, N, K, k_per_split);
  } else {
    dim3 grid((N + 63) / 64, (rows_ub + 3) / 4, splits);
    hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, (const float*)A, lda, (const float*)W, ldw, C, ldc,
                       split_stride, d_rows, N, K, k_per_split);
  }
  return hipGetLastError();
}
