// Matrix products C = A W^T for the rollout: activations A [rows, K] times
// weights W [N, K] (both K-contiguous), fp32 results, optional split over K.
//
// bf16 models: LDS-tiled gfx950 MFMA (v_mfma_f32_16x16x32_bf16).  A block
// owns a BM x BN output tile and walks its K range in BK = 64 steps: every
// thread fetches 16-byte pieces of the next A (hi and lo planes) and W tiles
// into registers while the waves multiply the current tiles out of LDS, then
// the pieces are written to LDS for the next step.  Each wave owns a WM x WN
// grid of 16 x 16 MFMA tiles.  The activation comes as hi/lo bf16 planes and
// every fragment takes two MFMAs (W*hi + W*lo) into one fp32 accumulator.
// Tile shapes are chosen by the row count: 16 rows for the decode tail up to
// 256 x 128 tiles for prefill.
//
// MFMA 16x16x32 lane layout: lane l supplies row (l % 16), k-slice
// 8*(l / 16) .. +7 of A and column (l % 16), the same k-slice of B; it
// receives C rows 4*(l / 16) .. +3 of column (l % 16).
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

constexpr int BK = 64;
constexpr int LDS_PAD = 8;             // bf16 elements of padding per LDS row
constexpr int LROW = BK + LDS_PAD;     // LDS row stride (elements)

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t lds_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(p));
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__((BM / (16 * WM)) * (BN / (16 * WN)) * 64) void k_gemm_tiled(
    const bf16_t* __restrict__ A, int lda, int64_t a_plane, const bf16_t* __restrict__ W, int ldw,
    float* __restrict__ C, int ldc, int64_t split_stride, const int* __restrict__ d_rows, int N, int K,
    int k_per_split) {
  constexpr int WAVES_M = BM / (16 * WM), WAVES_N = BN / (16 * WN);
  constexpr int NT = WAVES_M * WAVES_N * 64;
  constexpr int A_PIECES = BM * (BK / 8);          // 16-byte pieces per A plane tile
  constexpr int W_PIECES = BN * (BK / 8);
  static_assert((2 * A_PIECES) % NT == 0 && W_PIECES % NT == 0, "tile pieces must split evenly over threads");
  constexpr int A_PER_T = 2 * A_PIECES / NT;
  constexpr int W_PER_T = W_PIECES / NT;
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM * LROW];
  __shared__ __attribute__((aligned(16))) bf16_t sW[BN * LROW];

  const int M = *d_rows;
  const int m0 = blockIdx.y * BM;
  if (m0 >= M) return;
  const int n0 = blockIdx.x * BN;
  const int kb0 = blockIdx.z * k_per_split;
  const int ke = min(K, kb0 + k_per_split);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int lr = lane & 15, lk = (lane >> 4) * 8;

  u32x4_t ra[A_PER_T], rw[W_PER_T];
#define RG_FETCH(KK)                                                                                          \
  _Pragma("unroll") for (int i = 0; i < A_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int plane = p / A_PIECES, q = p % A_PIECES;                                                         \
    const int row = min(m0 + q / (BK / 8), M - 1); /* rows past M are computed, never stored */              \
    ra[i] = *reinterpret_cast<const u32x4_t*>(A + plane * a_plane + (int64_t)row * lda + (KK) + (q % (BK / 8)) * 8); \
  }                                                                                                           \
  _Pragma("unroll") for (int i = 0; i < W_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int col = min(n0 + p / (BK / 8), N - 1);                                                            \
    rw[i] = *reinterpret_cast<const u32x4_t*>(W + (int64_t)col * ldw + (KK) + (p % (BK / 8)) * 8);           \
  }
#define RG_STASH()                                                                                            \
  _Pragma("unroll") for (int i = 0; i < A_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int plane = p / A_PIECES, q = p % A_PIECES;                                                         \
    *reinterpret_cast<u32x4_t*>(&sA[plane][(q / (BK / 8)) * LROW + (q % (BK / 8)) * 8]) = ra[i];             \
  }                                                                                                           \
  _Pragma("unroll") for (int i = 0; i < W_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    *reinterpret_cast<u32x4_t*>(&sW[(p / (BK / 8)) * LROW + (p % (BK / 8)) * 8]) = rw[i];                    \
  }

  f32x4_t acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (kb0 < ke) {
    RG_FETCH(kb0)
    for (int k = kb0; k < ke; k += BK) {
      __syncthreads();          // the previous step's fragment reads are done
      RG_STASH()
      __syncthreads();
      if (k + BK < ke) { RG_FETCH(k + BK) }   // next tiles in flight while this one is multiplied
#pragma unroll
      for (int ks = 0; ks < BK; ks += 32) {
        bf16x8_t bw[WN];
#pragma unroll
        for (int j = 0; j < WN; ++j) bw[j] = lds_frag(&sW[((wn * WN + j) * 16 + lr) * LROW + ks + lk]);
#pragma unroll
        for (int i = 0; i < WM; ++i) {
          const int arow = (wm * WM + i) * 16 + lr;
          const bf16x8_t ah = lds_frag(&sA[0][arow * LROW + ks + lk]);
          const bf16x8_t al = lds_frag(&sA[1][arow * LROW + ks + lk]);
#pragma unroll
          for (int j = 0; j < WN; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bw[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bw[j], acc[i][j], 0, 0, 0);
          }
        }
      }
    }
  }
#undef RG_FETCH
#undef RG_STASH
  float* cp = C + blockIdx.z * split_stride;
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) {
      const int col = n0 + (wn * WN + j) * 16 + lr;
      if (col >= N) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = m0 + (wm * WM + i) * 16 + (lane >> 4) * 4 + e;
        if (r < M) cp[(int64_t)r * ldc + col] = acc[i][j][e];
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

template <int BM, int BN, int WM, int WN>
hipError_t launch_tiled(const void* A, int lda, int64_t a_plane, const void* W, int ldw, float* C, int ldc,
                        int64_t split_stride, const int* d_rows, int rows_ub, int N, int K, int splits,
                        int k_per_split, hipStream_t st) {
  constexpr int NT = (BM / (16 * WM)) * (BN / (16 * WN)) * 64;
  dim3 grid((N + BN - 1) / BN, (rows_ub + BM - 1) / BM, splits);
  hipLaunchKernelGGL((k_gemm_tiled<BM, BN, WM, WN>), grid, dim3(NT), 0, st, (const bf16_t*)A, lda, a_plane,
                     (const bf16_t*)W, ldw, C, ldc, split_stride, d_rows, N, K, k_per_split);
  return hipGetLastError();
}

}  // namespace

int gemm_tile_rows(int dtype, int rows_ub) {
  if (dtype != 1) return 4;
  if (rows_ub <= 16) return 16;
  if (rows_ub <= 32) return 32;
  if (rows_ub <= 64) return 64;
  if (rows_ub <= 128) return 128;
  return 256;
}

int gemm_tile_cols(int dtype, int rows_ub) { return dtype == 1 ? 128 : 64; }

hipError_t launch_gemm(int dtype, const void* A, int lda, int64_t a_plane, const void* W, int ldw, float* C, int ldc,
                       int64_t split_stride, const int* d_rows, int rows_ub, int N, int K, int splits,
                       int k_per_split, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if (dtype == 1) {
    if (K % BK || k_per_split % BK || N % 16) return hipErrorInvalidValue;
    switch (gemm_tile_rows(dtype, rows_ub)) {
      case 16: return launch_tiled<16, 128, 1, 2>(A, lda, a_plane, W, ldw, C, ldc, split_stride, d_rows, rows_ub, N, K, splits, k_per_split, st);
      case 32: return launch_tiled<32, 128, 1, 4>(A, lda, a_plane, W, ldw, C, ldc, split_stride, d_rows, rows_ub, N, K, splits, k_per_split, st);
      case 64: return launch_tiled<64, 128, 2, 4>(A, lda, a_plane, W, ldw, C, ldc, split_stride, d_rows, rows_ub, N, K, splits, k_per_split, st);
      case 128: return launch_tiled<128, 128, 4, 4>(A, lda, a_plane, W, ldw, C, ldc, split_stride, d_rows, rows_ub, N, K, splits, k_per_split, st);
      default: return launch_tiled<256, 128, 4, 4>(A, lda, a_plane, W, ldw, C, ldc, split_stride, d_rows, rows_ub, N, K, splits, k_per_split, st);
    }
  }
  dim3 grid((N + 63) / 64, (rows_ub + 3) / 4, splits);
  hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, (const float*)A, lda, (const float*)W, ldw, C, ldc,
                     split_stride, d_rows, N, K, k_per_split);
  return hipGetLastError();
}
