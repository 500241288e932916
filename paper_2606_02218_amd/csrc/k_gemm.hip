// Matrix products of the decoder, y = x W^T with activations [rows, K] and
// weights W [N, K] (both K-contiguous), each with a fused epilogue:
//   STORE     C[r][n] = y                          (lm head logits)
//   RESIDUAL  x[r][n] += y                         (O and down projections)
//   SWIGLU    act[r][f] = silu(gate) * up          (gate/up projection; packed
//             columns come as [16 gate | 16 up] per 32)
//   QKV       RoPE on the query and key heads; q -> fp32 buffer, k and v ->
//             the row's KV page (keys as [slot][dim], values as [dim][slot]).
//             Within each head the packed weight rows come in 16-row tiles
//             ordered (dims 0-15, dims h/2..h/2+15, dims 16-31, ...) so that
//             a rotated pair (d, d + h/2) lies in adjacent column tiles.
//
// bf16 models: LDS-tiled gfx950 MFMA (v_mfma_f32_16x16x32_bf16).  A block
// owns a BM x BN output tile and walks its K range in BK = 64 steps: every
// thread fetches 16-byte pieces of the next A (hi and lo planes) and W tiles
// into registers while the waves multiply the current tiles out of LDS, then
// the pieces are written to LDS for the next step.  Each wave owns a WM x WN
// grid of 16 x 16 MFMA tiles.  The activation comes as hi/lo bf16 planes and
// every fragment takes two MFMAs (W*hi + W*lo) into one fp32 accumulator.
//
// Split over K: the grid's z dimension splits K and every split writes its
// fp32 partial; k_split_epilogue then sums the partials in split order (one
// block per row and 128 columns) and runs the epilogue.  Without a split the
// epilogue runs straight from the accumulators.
//
// MFMA 16x16x32 lane layout: lane l supplies row (l % 16), k-slice
// 8*(l / 16) .. +7 of A and column (l % 16), the same k-slice of B; it
// receives C rows 4*(l / 16) .. +3 of column (l % 16).
#include "rg_device.h"
#include "rg_kernels.h"

namespace {

constexpr int BK_MAX = 64;             // K step of the small tiles; large tiles may use 32
constexpr int LDS_PAD = 16;            // bf16 elements of padding per LDS row (rows 160 B apart: no bank conflicts)

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t lds_frag(const bf16_t* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(p));
}

template <typename KV>
__device__ __forceinline__ void kv_store(KV* p, float v);
template <> __device__ __forceinline__ void kv_store<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void kv_store<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// Sum of the split partials of element (r, c), in split order.  The loads
// of a batch of 16 splits are all issued before its first add.
__device__ __forceinline__ float split_sum(const GemmEpi& ep, int S, int64_t off) {
  constexpr int BATCH = 16;
  const float* p = ep.part + off;
  const int64_t st = ep.part_stride;
  float acc = 0.f;
  for (int s0 = 0; s0 < S; s0 += BATCH) {
    float v[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) v[j] = s0 + j < S ? p[(s0 + j) * st] : 0.f;
#pragma unroll
    for (int j = 0; j < BATCH; ++j) acc += v[j];
  }
  return acc;
}

// QKV epilogue of row r for packed column c (a lower-half tile column: bit 4
// of c is 0) holding dim d of its head, and c + 16 holding dim d + half.
template <typename KV>
__device__ __forceinline__ void qkv_store(const GemmEpi& ep, int r, int c, float a, float b) {
  const int hd = ep.hd, half = hd / 2;
  const int head = c / hd, p = c % hd;
  const int d = (p >> 5) * 16 + (p & 15);
  const int pos = ep.row_pos[r];
  KV* pool = (KV*)ep.kv_pool;
  if (head >= ep.n_q + ep.n_kv) {                     // value head: no rotation, V^T layout
    const int kvh = head - ep.n_q - ep.n_kv;
    const int page = ep.page_tab[(int64_t)ep.row_tab[r] * ep.tab_stride + pos / 16];
    KV* vb = pool + (int64_t)page * ep.geom.page_stride + (int64_t)ep.layer * ep.geom.layer_stride +
             ((int64_t)ep.n_kv + kvh) * 16 * hd;
    kv_store<KV>(vb + kv_v_off(pos & 15, d, hd), a);
    kv_store<KV>(vb + kv_v_off(pos & 15, d + half, hd), b);
    return;
  }
  const float co = ep.rope_cos[(int64_t)pos * half + d], si = ep.rope_sin[(int64_t)pos * half + d];
  const float ra = a * co - b * si, rb = b * co + a * si;
  if (head < ep.n_q) {
    float* qo = ep.q_out + ((int64_t)r * ep.n_q + head) * hd;
    qo[d] = ra;
    qo[d + half] = rb;
  } else {
    const int kvh = head - ep.n_q;
    const int page = ep.page_tab[(int64_t)ep.row_tab[r] * ep.tab_stride + pos / 16];
    KV* kp = pool + (int64_t)page * ep.geom.page_stride + (int64_t)ep.layer * ep.geom.layer_stride +
             (int64_t)kvh * 16 * hd;
    kv_store<KV>(kp + kv_k_off(pos & 15, d), ra);
    kv_store<KV>(kp + kv_k_off(pos & 15, d + half), rb);
  }
}

// QKV epilogue straight from the accumulators of one wave (rows
// m0 + (wm*WM + i)*16 + 4*(lane/16) + e, column tiles wn*WN + j).  One row
// block i at a time, every load it needs (row position, KV page, the RoPE
// cos/sin of each rotated pair) is issued before the first store: through
// restrict-qualified pointers the loads of a block do not wait on the stores
// of the previous one, so the tile pays a few load latencies instead of one
// per element.
template <int WM, int WN>
__device__ __forceinline__ void qkv_tile_store(const f32x4_t (&acc)[WM][WN], const GemmEpi& ep, int m0, int n0, int M,
                                               int N, int wm, int wn, int lane,
                                               const int32_t* __restrict__ row_pos,
                                               const int32_t* __restrict__ row_tab,
                                               const int32_t* __restrict__ page_tab,
                                               const float* __restrict__ rcos, const float* __restrict__ rsin,
                                               float* __restrict__ q_out, bf16_t* __restrict__ pool) {
  const int lr = lane & 15;
  const int hd = ep.hd, half = hd / 2, n_rot = ep.n_q + ep.n_kv;
#pragma unroll
  for (int i = 0; i < WM; ++i) {
    const int rb = m0 + (wm * WM + i) * 16 + (lane >> 4) * 4;
    int pos[4];
    int64_t kvb[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = min(rb + e, M - 1);
      pos[e] = row_pos[r];
      const int page = page_tab[(int64_t)row_tab[r] * ep.tab_stride + pos[e] / 16];
      kvb[e] = (int64_t)page * ep.geom.page_stride + (int64_t)ep.layer * ep.geom.layer_stride;
    }
    float co[WN / 2][4], si[WN / 2][4];
#pragma unroll
    for (int j = 0; j < WN; j += 2) {
      const int c = min(n0 + (wn * WN + j) * 16 + lr, N - 1);
      const int p = c % hd, d = (p >> 5) * 16 + (p & 15);
      const bool rot = c / hd < n_rot;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        co[j / 2][e] = rot ? rcos[(int64_t)pos[e] * half + d] : 1.f;
        si[j / 2][e] = rot ? rsin[(int64_t)pos[e] * half + d] : 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < WN; j += 2) {
      const int c = n0 + (wn * WN + j) * 16 + lr;   // lower tile's column
      if (c >= N) continue;
      const int head = c / hd, p = c % hd, d = (p >> 5) * 16 + (p & 15);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (rb + e >= M) continue;
        const float a = acc[i][j][e], b = acc[i][j + 1][e];
        const int slot = pos[e] & 15;
        if (head >= n_rot) {                               // value head: V^T layout, no rotation
          bf16_t* vb = pool + kvb[e] + ((int64_t)ep.n_kv + head - n_rot) * 16 * hd;
          vb[kv_v_off(slot, d, hd)] = f32_to_bf16(a);
          vb[kv_v_off(slot, d + half, hd)] = f32_to_bf16(b);
          continue;
        }
        const float ra = a * co[j / 2][e] - b * si[j / 2][e], rr = b * co[j / 2][e] + a * si[j / 2][e];
        if (head < ep.n_q) {
          float* qo = q_out + ((int64_t)(rb + e) * ep.n_q + head) * hd;
          qo[d] = ra;
          qo[d + half] = rr;
        } else {
          bf16_t* kp = pool + kvb[e] + (int64_t)(head - ep.n_q) * 16 * hd;
          kp[kv_k_off(slot, d)] = f32_to_bf16(ra);
          kp[kv_k_off(slot, d + half)] = f32_to_bf16(rr);
        }
      }
    }
  }
}

// Epilogue of a finished tile whose split partials are in ep.part: rows
// m0..m0+BM-1, columns n0..n0+BN-1 (< N); only rows below M are stored.
// STORE, RESIDUAL and SWIGLU sum the partials of every row of the tile (all
// inside the partial buffer; columns past N read a column in range) before
// testing row and column, so their loads wait neither for the row count nor
// for a test of a kernel argument; QKV needs the row's position and page and
// tests first.  Every thread of the block calls it.
template <int EPI, int BM, int BN, int NT, int SPLIT, typename KV>
__device__ void tile_epilogue(const GemmEpi& ep, int S, int m0, int n0, int M, int N, int tid) {
  if constexpr (EPI == GEMM_EPI_STORE || EPI == GEMM_EPI_RESIDUAL) {
    for (int i = tid; i < BM * BN; i += NT) {
      const int r = m0 + i / BN, c = n0 + i % BN;
      const float v = split_sum(ep, S, (int64_t)r * N + min(c, N - 1));
      if (r >= M || c >= N) continue;
      if constexpr (EPI == GEMM_EPI_STORE) ep.C[(int64_t)r * ep.ldc + c] = v;
      else ep.x[(int64_t)r * ep.ldx + c] += v;
    }
  } else if constexpr (EPI == GEMM_EPI_SWIGLU) {
    for (int i = tid; i < BM * (BN / 2); i += NT) {
      const int r = m0 + i / (BN / 2), q = i % (BN / 2);
      const int gc = n0 + (q >> 4) * 32 + (q & 15);    // gate column; up is 16 further
      const int gl = min(gc, N - 17);                    // gc itself while in range (N % 32 == 0)
      const float gt = split_sum(ep, S, (int64_t)r * N + gl);
      const float up = split_sum(ep, S, (int64_t)r * N + gl + 16);
      if (r >= M || gc >= N) continue;
      act_store<SPLIT>(ep.act, (int64_t)r * ep.act_ld + (gc >> 5) * 16 + (q & 15), gt / (1.0f + expf(-gt)) * up);
    }
  } else {  // GEMM_EPI_QKV: packed columns; a lower-half tile owns the rotated pair
    for (int i = tid; i < BM * BN; i += NT) {
      const int r = m0 + i / BN, c = n0 + i % BN;
      if (r >= M || c >= N || ((c >> 4) & 1)) continue;
      const int64_t roff = (int64_t)r * N;
      qkv_store<KV>(ep, r, c, split_sum(ep, S, roff + c), split_sum(ep, S, roff + c + 16));
    }
  }
}

// A 16-byte piece of W.  NT: a non-temporal load, for weights that no other
// block of the launch reads (one row tile): streamed through without
// claiming cache space, which measured 6.5-6.7 TB/s against 5.9-6.1 TB/s
// for plain loads in a pure streaming read of 8 GiB.
__device__ __forceinline__ int k_split_count(int K, int k_per_split) { return (K + k_per_split - 1) / k_per_split; }

template <bool NT>
__device__ __forceinline__ u32x4_t load_w(const bf16_t* p) {
  if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  else return *reinterpret_cast<const u32x4_t*>(p);
}

template <int BM, int BN, int WM, int WN, int STAGES, int BK, int EPI, bool NTW, bool XO>
__global__ __launch_bounds__((BM / (16 * WM)) * (BN / (16 * WN)) * 64) void k_gemm_tiled(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, const int* __restrict__ d_rows, int64_t a_plane,
    int lda, int ldw, int rows_cap, int N, int K, int k_per_split, int gx, int gy, GemmEpi ep) {
  // The arguments the first loads need come first (14 dwords, which the
  // build preloads into scalar registers at dispatch).  The row count is
  // read first but waited for only after the first K step's loads are
  // issued: those clamp A rows to the launch's row bound rows_cap (>= the
  // count; the activation buffer holds that many rows), so they do not
  // depend on it.  Rows past the count are multiplied, never stored.
  const int rows_now = *d_rows;
  constexpr int WAVES_M = BM / (16 * WM), WAVES_N = BN / (16 * WN);
  constexpr int NT = WAVES_M * WAVES_N * 64;
  constexpr int LROW = BK + LDS_PAD;                // LDS row stride (elements)
  static_assert(BK == 32 || BK == 64, "K step");
  constexpr int A_PIECES = BM * (BK / 8);          // 16-byte pieces per A plane tile
  constexpr int W_PIECES = BN * (BK / 8);
  static_assert((2 * A_PIECES) % NT == 0 && W_PIECES % NT == 0, "tile pieces must split evenly over threads");
  static_assert((EPI != GEMM_EPI_SWIGLU && EPI != GEMM_EPI_QKV) || WN % 2 == 0, "pairs of adjacent column tiles");
  constexpr int A_PER_T = 2 * A_PIECES / NT;
  constexpr int W_PER_T = W_PIECES / NT;
  __shared__ __attribute__((aligned(16))) bf16_t sA[2][BM * LROW];
  __shared__ __attribute__((aligned(16))) bf16_t sW[BN * LROW];

  int tx = blockIdx.x, ty = blockIdx.y, tz = blockIdx.z;
  if constexpr (XO) {
    // A 1-D grid of a multiple of 8 blocks, dealt to the 8 XCDs in turn:
    // XCD x = b % 8 takes the contiguous tile range [x*per, (x+1)*per)
    // (split-major), walked in groups of TILE_GROUP row tiles.  Within a
    // group the row tiles of one column tile are consecutive, so the blocks
    // that an XCD runs at once share A rows and W columns in its L2.
    constexpr int TILE_GROUP = 4;
    const int per = gridDim.x / 8;
    int w = (blockIdx.x % 8) * per + blockIdx.x / 8;
    if (w >= gx * gy * (int)k_split_count(K, k_per_split)) return;
    tz = w / (gx * gy);
    w -= tz * gx * gy;
    const int gsz = TILE_GROUP * gx;                    // tiles per full group
    const int g = w / gsz, r0 = g * TILE_GROUP;
    const int rows_g = min(TILE_GROUP, gy - r0);       // the last group may be short
    const int wi = w - g * gsz;
    ty = r0 + wi % rows_g;
    tx = wi / rows_g;
  }
  const int m0 = ty * BM;   // < rows_cap: the grid has ceil(rows_cap / BM) row tiles
  const int n0 = tx * BN;
  const int kb0 = tz * k_per_split;
  const int ke = min(K, kb0 + k_per_split);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int lr = lane & 15, lk = (lane >> 4) * 8;

  // STAGES register sets: the global loads of step k + STAGES*BK are issued
  // right after step k's tiles reach LDS, so STAGES steps of loads are in
  // flight while one step is multiplied out (HBM latency exceeds one step of
  // MFMA work by a wide margin).
  u32x4_t ra[STAGES][A_PER_T], rw[STAGES][W_PER_T];
#define RG_FETCH(S, KK)                                                                                       \
  _Pragma("unroll") for (int i = 0; i < A_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int plane = p / A_PIECES, q = p % A_PIECES;                                                         \
    const int row = min(m0 + q / (BK / 8), rows_cap - 1); /* rows past M are computed, never stored */       \
    ra[S][i] = *reinterpret_cast<const u32x4_t*>(A + plane * a_plane + (int64_t)row * lda + (KK) + (q % (BK / 8)) * 8); \
  }                                                                                                           \
  _Pragma("unroll") for (int i = 0; i < W_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int col = min(n0 + p / (BK / 8), N - 1);                                                            \
    rw[S][i] = load_w<NTW>(W + (int64_t)col * ldw + (KK) + (p % (BK / 8)) * 8);                               \
  }
#define RG_STASH(S)                                                                                           \
  _Pragma("unroll") for (int i = 0; i < A_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    const int plane = p / A_PIECES, q = p % A_PIECES;                                                         \
    *reinterpret_cast<u32x4_t*>(&sA[plane][(q / (BK / 8)) * LROW + (q % (BK / 8)) * 8]) = ra[S][i];          \
  }                                                                                                           \
  _Pragma("unroll") for (int i = 0; i < W_PER_T; ++i) {                                                       \
    const int p = tid + i * NT;                                                                               \
    *reinterpret_cast<u32x4_t*>(&sW[(p / (BK / 8)) * LROW + (p % (BK / 8)) * 8]) = rw[S][i];                 \
  }

  f32x4_t acc[WM][WN];
#pragma unroll
  for (int i = 0; i < WM; ++i)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int s = 0; s < STAGES; ++s)
    if (kb0 + s * BK < ke) { RG_FETCH(s, kb0 + s * BK) }
  // keeps the loads above in front of the row-count test (no sinking past it)
  __asm__ volatile("" ::: "memory");
  const int M = min(rows_now, rows_cap);
  if (m0 >= M) return;
  for (int k = kb0; k < ke; k += STAGES * BK) {
#pragma unroll
    for (int s = 0; s < STAGES; ++s) {
      const int kk = k + s * BK;
      if (kk < ke) {
        __syncthreads();          // the previous step's fragment reads are done
        RG_STASH(s)
        __syncthreads();
        if (kk + STAGES * BK < ke) { RG_FETCH(s, kk + STAGES * BK) }
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
  }
#undef RG_FETCH
#undef RG_STASH

  if constexpr (EPI == GEMM_EPI_PARTIAL) {
    float* pp = ep.part + tz * ep.part_stride;
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = n0 + (wn * WN + j) * 16 + lr;
        if (col >= N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = m0 + (wm * WM + i) * 16 + (lane >> 4) * 4 + e;
          if (r < M) pp[(int64_t)r * N + col] = acc[i][j][e];
        }
      }
  } else if constexpr (EPI == GEMM_EPI_QKV) {
    qkv_tile_store<WM, WN>(acc, ep, m0, n0, M, N, wm, wn, lane, ep.row_pos, ep.row_tab, ep.page_tab, ep.rope_cos,
                           ep.rope_sin, ep.q_out, (bf16_t*)ep.kv_pool);
  } else if constexpr (EPI == GEMM_EPI_SWIGLU) {
    // tiles 2m and 2m+1 of a wave pair up: (gate, up)
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; j += 2) {
        const int c = n0 + (wn * WN + j) * 16 + lr;   // lower tile's column
        if (c >= N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = m0 + (wm * WM + i) * 16 + (lane >> 4) * 4 + e;
          if (r >= M) continue;
          const float a = acc[i][j][e], b = acc[i][j + 1][e];
          act_store<1>(ep.act, (int64_t)r * ep.act_ld + (c >> 5) * 16 + lr, a / (1.0f + expf(-a)) * b);
        }
      }
  } else {
    float* cp = EPI == GEMM_EPI_RESIDUAL ? ep.x : ep.C;
    const int ld = EPI == GEMM_EPI_RESIDUAL ? ep.ldx : ep.ldc;
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = n0 + (wn * WN + j) * 16 + lr;
        if (col >= N) continue;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = m0 + (wm * WM + i) * 16 + (lane >> 4) * 4 + e;
          if (r < M) {
            if constexpr (EPI == GEMM_EPI_RESIDUAL) cp[(int64_t)r * ld + col] += acc[i][j][e];
            else cp[(int64_t)r * ld + col] = acc[i][j][e];
          }
        }
      }
  }
}

// Residual add of the split partials followed by the next RMSNorm of the row
// (x += sum_s part_s; act = x / sqrt(mean(x^2) + eps) * g): one 1024-thread
// block per row, thread t owning columns t + 1024 k (k < CPT).  A thread issues
// its x and g loads and a batch of its split partials before the first add,
// and the row stays in registers between the sum of squares and the store.
// The sums run in split order, as in split_sum.
template <int SPLIT, int CPT>
__global__ __launch_bounds__(1024) void k_split_residual_norm(const int* __restrict__ d_rows,
                                                               const float* __restrict__ part, int64_t pst,
                                                               float* __restrict__ x, const float* __restrict__ norm_g,
                                                               int N, int S, int ldx, GemmEpi ep) {
  constexpr int NT = 1024;
  constexpr int BATCH = CPT <= 2 ? 16 : 32 / CPT;   // splits loaded per batch
  const int r = blockIdx.x;
  // Blocks of rows past the count (r < the launch's row bound, inside every
  // buffer) run the same loads and sums but store nothing, so no load waits
  // for the count.
  const int rows_now = *d_rows;
  __shared__ float red[16];
  float* xr = x + (int64_t)r * ldx;
  const float* pr = part + (int64_t)r * N;
  float xv[CPT], gv[CPT], acc[CPT];
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    const int c = threadIdx.x + k * NT;
    xv[k] = c < N ? xr[c] : 0.f;
    gv[k] = c < N ? norm_g[c] : 0.f;
    acc[k] = 0.f;
  }
  for (int s0 = 0; s0 < S; s0 += BATCH) {
    float t[BATCH][CPT];
#pragma unroll
    for (int j = 0; j < BATCH; ++j)
#pragma unroll
      for (int k = 0; k < CPT; ++k) {
        const int c = threadIdx.x + k * NT;
        t[j][k] = (s0 + j < S && c < N) ? pr[(s0 + j) * pst + c] : 0.f;
      }
#pragma unroll
    for (int j = 0; j < BATCH; ++j)
#pragma unroll
      for (int k = 0; k < CPT; ++k) acc[k] += t[j][k];
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    xv[k] += acc[k];
    ss = fmaf(xv[k], xv[k], ss);
  }
  ss = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)N + ep.norm_eps);
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    const int c = threadIdx.x + k * NT;
    if (c < N && r < rows_now) {
      xr[c] = xv[k];
      act_store<SPLIT>(ep.norm_out, (int64_t)r * N + c, xv[k] * inv * gv[k]);
    }
  }
}

// QKV epilogue of split partials for bf16 models, 16 bytes at a time: thread
// u of row r owns packed columns c..c+3 (c = 32 (u / 4) + 4 (u % 4), in the
// lower half of a 32-column group) and their rotation partners c+16..c+19.
// The partials of both column quads are summed in split order (as split_sum),
// rotated, and written as one 16-byte q piece per half or one 8-byte key piece
// per half (values: their transposed layout, one element at a time).  Same
// arithmetic as qkv_store; one wave per 64 quads of a row.
__global__ __launch_bounds__(64) void k_qkv_epilogue4(const int* __restrict__ d_rows, const float* __restrict__ part,
                                                      int64_t pst, int N, int S, GemmEpi ep) {
  typedef float f4 __attribute__((ext_vector_type(4)));
  constexpr int BATCH = 16;
  const int r = blockIdx.y;
  const int u = blockIdx.x * 64 + threadIdx.x;
  const int rows_now = *d_rows;   // waited for after the partials' loads
  __builtin_assume(S >= 1);
  const int uc = min(u, N / 8 - 1);   // a quad in range: u's own test comes after the loads
  const int c = (uc >> 2) * 32 + (uc & 3) * 4;
  const int hd = ep.hd, half = hd / 2;
  const int head = c / hd, p = c % hd, d = (p >> 5) * 16 + (p & 15);
  const f4* pr = reinterpret_cast<const f4*>(part + (int64_t)r * N + c);
  const int64_t pst4 = pst / 4;
  f4 a = {0.f, 0.f, 0.f, 0.f}, b = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < S; s0 += BATCH) {
    f4 ta[BATCH], tb[BATCH];
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      ta[j] = s0 + j < S ? pr[(s0 + j) * pst4] : f4{0.f, 0.f, 0.f, 0.f};
      tb[j] = s0 + j < S ? pr[(s0 + j) * pst4 + 4] : f4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < BATCH; ++j) {
      a += ta[j];
      b += tb[j];
    }
  }
  // a row past the count has no position or page yet
  if (r >= rows_now || u >= N / 8) return;
  const int pos = ep.row_pos[r];
  bf16_t* pool = (bf16_t*)ep.kv_pool;
  const int n_rot = ep.n_q + ep.n_kv;
  if (head >= n_rot) {                               // value head: no rotation, V^T layout
    const int page = ep.page_tab[(int64_t)ep.row_tab[r] * ep.tab_stride + pos / 16];
    bf16_t* vb = pool + (int64_t)page * ep.geom.page_stride + (int64_t)ep.layer * ep.geom.layer_stride +
                 ((int64_t)ep.n_kv + head - n_rot) * 16 * hd;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      vb[kv_v_off(pos & 15, d + e, hd)] = f32_to_bf16(a[e]);
      vb[kv_v_off(pos & 15, d + e + half, hd)] = f32_to_bf16(b[e]);
    }
    return;
  }
  const f4 co = *reinterpret_cast<const f4*>(ep.rope_cos + (int64_t)pos * half + d);
  const f4 si = *reinterpret_cast<const f4*>(ep.rope_sin + (int64_t)pos * half + d);
  f4 ra, rb;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    ra[e] = a[e] * co[e] - b[e] * si[e];
    rb[e] = b[e] * co[e] + a[e] * si[e];
  }
  if (head < ep.n_q) {
    float* qo = ep.q_out + ((int64_t)r * ep.n_q + head) * hd;
    *reinterpret_cast<f4*>(qo + d) = ra;
    *reinterpret_cast<f4*>(qo + d + half) = rb;
  } else {
    const int page = ep.page_tab[(int64_t)ep.row_tab[r] * ep.tab_stride + pos / 16];
    bf16_t* kp = pool + (int64_t)page * ep.geom.page_stride + (int64_t)ep.layer * ep.geom.layer_stride +
                 (int64_t)(head - ep.n_q) * 16 * hd;
    uint2 ka, kb;
    ka.x = (uint32_t)f32_to_bf16(ra[0]) | ((uint32_t)f32_to_bf16(ra[1]) << 16);
    ka.y = (uint32_t)f32_to_bf16(ra[2]) | ((uint32_t)f32_to_bf16(ra[3]) << 16);
    kb.x = (uint32_t)f32_to_bf16(rb[0]) | ((uint32_t)f32_to_bf16(rb[1]) << 16);
    kb.y = (uint32_t)f32_to_bf16(rb[2]) | ((uint32_t)f32_to_bf16(rb[3]) << 16);
    *reinterpret_cast<uint2*>(kp + kv_k_off(pos & 15, d)) = ka;
    *reinterpret_cast<uint2*>(kp + kv_k_off(pos & 15, d + half)) = kb;
  }
}

// Sum of split partials + epilogue: one block of 128 threads per (128
// columns, row).  SPLIT: activation output as hi/lo bf16 planes.
template <int EPI, int SPLIT, typename KV>
__global__ __launch_bounds__(128) void k_split_epilogue(const int* __restrict__ d_rows, float* __restrict__ part,
                                                        int64_t pst, int N, int S, GemmEpi ep) {
  const int r = blockIdx.y;
  const int rows_now = *d_rows;
  ep.part = part;          // the preloaded copies
  ep.part_stride = pst;
  if constexpr (EPI == GEMM_EPI_QKV) {
    if (r >= rows_now) return;
  }
  tile_epilogue<EPI, 1, 128, 128, SPLIT, KV>(ep, S, r, blockIdx.x * 128, rows_now, N, threadIdx.x);
}

// fp32 models: plain fp32 FMA, one thread per output, 64 columns x 4 rows per
// block, into the partial buffer; k_split_epilogue then runs the epilogue.
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const float* __restrict__ W, int ldw,
                                                  float* __restrict__ C, const int* __restrict__ d_rows, int N,
                                                  int K) {
  const int M = *d_rows;
  const int r = blockIdx.y * 4 + (threadIdx.x >> 6);
  const int n = blockIdx.x * 64 + (threadIdx.x & 63);
  if (r >= M || n >= N) return;
  const float* a = A + (int64_t)r * lda;
  const float* w = W + (int64_t)n * ldw;
  float acc = 0.f;
  for (int k = 0; k < K; ++k) acc = fmaf(a[k], w[k], acc);
  C[(int64_t)r * N + n] = acc;
}

template <int BM, int BN, int WM, int WN, int STAGES, int BK = 64>
hipError_t launch_tiled(const void* A, int lda, int64_t a_plane, const void* W, int ldw, const int* d_rows,
                        int rows_ub, int N, int K, int splits, int k_per_split, const GemmEpi& ep, hipStream_t st) {
  constexpr int NT = (BM / (16 * WM)) * (BN / (16 * WN)) * 64;
  const int gx = (N + BN - 1) / BN, gy = (rows_ub + BM - 1) / BM;
  dim3 grid(gx, gy, splits);
  // The XCD-aware grouped tile order for 256 x 256 tiles, and for wide
  // outputs (gate/up) read by 8 or more row tiles: there the default order
  // fetches each weight tile about 7 times per launch from beyond L2 (gate/up
  // at 512 rows: 418 MB of L2 misses for 58 MB of operands, against 120 MB
  // in this order, 7 % faster).  For the narrow outputs at 256-512 rows it
  // measured 2-9 % slower, so they keep the default order.
  const int order1d = BM == 256 || (N >= 8192 && gy >= 8);
  if (order1d) {
    if ((K + k_per_split - 1) / k_per_split != splits) return hipErrorInvalidValue;
    grid = dim3((unsigned)(((int64_t)gx * gy * splits + 7) / 8 * 8));
  }
  // One row tile: every weight piece is read by one block only, so its loads
  // are non-temporal.  With several row tiles the weight tiles are re-read
  // by the other row tiles' blocks through L2, and non-temporal loads there
  // measured 12 % slower over the 1.5B group step.
  const bool ntw = gy == 1;
  // The tile order is a template parameter, so that no kernel argument
  // decides a branch ahead of the first loads.  Below 256 x 256 tiles the
  // grouped order needs 8 or more row tiles, so it never meets ntw.
#define RG_TILED_K(E, NTV, XOV)                                                                               \
  hipLaunchKernelGGL((k_gemm_tiled<BM, BN, WM, WN, STAGES, BK, E, NTV, XOV>), grid, dim3(NT), 0, st,           \
                     (const bf16_t*)A, (const bf16_t*)W, d_rows, a_plane, lda, ldw, rows_ub, N, K, k_per_split, gx, \
                     gy, ep)
#define RG_TILED(E)                                                                                           \
  do {                                                                                                        \
    if constexpr (BM == 256) {                                                                                \
      if (ntw) RG_TILED_K(E, true, true);                                                                     \
      else RG_TILED_K(E, false, true);                                                                        \
    } else {                                                                                                  \
      if (order1d) RG_TILED_K(E, false, true);                                                                \
      else if (ntw) RG_TILED_K(E, true, false);                                                               \
      else RG_TILED_K(E, false, false);                                                                       \
    }                                                                                                         \
  } while (0)
  if (splits > 1) {
    RG_TILED(GEMM_EPI_PARTIAL);
  } else {
    switch (ep.mode) {
      case GEMM_EPI_STORE: RG_TILED(GEMM_EPI_STORE); break;
      case GEMM_EPI_RESIDUAL: RG_TILED(GEMM_EPI_RESIDUAL); break;
      case GEMM_EPI_SWIGLU: RG_TILED(GEMM_EPI_SWIGLU); break;
      case GEMM_EPI_QKV: RG_TILED(GEMM_EPI_QKV); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef RG_TILED
#undef RG_TILED_K
  return hipGetLastError();
}

template <int SPLIT, typename KV>
hipError_t launch_split_epilogue(const int* d_rows, int rows_ub, int N, int S, const GemmEpi& ep, hipStream_t st) {
  if (ep.mode == GEMM_EPI_RESIDUAL && ep.norm_g) {
    const int cpt = (N + 1023) / 1024;
#define RG_SRN(C)                                                                                             \
  hipLaunchKernelGGL((k_split_residual_norm<SPLIT, C>), dim3(rows_ub), dim3(1024), 0, st, d_rows, ep.part,        \
                     ep.part_stride, ep.x, ep.norm_g, N, S, ep.ldx, ep)
    if (cpt <= 1) RG_SRN(1);
    else if (cpt <= 2) RG_SRN(2);
    else if (cpt <= 4) RG_SRN(4);
    else if (cpt <= 8) RG_SRN(8);
    else return hipErrorInvalidValue;   // rows wider than 8192
#undef RG_SRN
    return hipGetLastError();
  }
  if constexpr (SPLIT == 1) {
    if (ep.mode == GEMM_EPI_QKV && N % 32 == 0 && ep.hd % 32 == 0 && ep.part_stride % 4 == 0) {
      hipLaunchKernelGGL(k_qkv_epilogue4, dim3((N / 8 + 63) / 64, rows_ub), dim3(64), 0, st, d_rows, ep.part,
                         ep.part_stride, N, S, ep);
      return hipGetLastError();
    }
  }
  dim3 grid((N + 127) / 128, rows_ub);
  switch (ep.mode) {
    case GEMM_EPI_STORE:
      hipLaunchKernelGGL((k_split_epilogue<GEMM_EPI_STORE, SPLIT, KV>), grid, dim3(128), 0, st, d_rows, ep.part,
                         ep.part_stride, N, S, ep);
      break;
    case GEMM_EPI_RESIDUAL:
      hipLaunchKernelGGL((k_split_epilogue<GEMM_EPI_RESIDUAL, SPLIT, KV>), grid, dim3(128), 0, st, d_rows, ep.part,
                         ep.part_stride, N, S, ep);
      break;
    case GEMM_EPI_SWIGLU:
      hipLaunchKernelGGL((k_split_epilogue<GEMM_EPI_SWIGLU, SPLIT, KV>), grid, dim3(128), 0, st, d_rows, ep.part,
                         ep.part_stride, N, S, ep);
      break;
    case GEMM_EPI_QKV:
      hipLaunchKernelGGL((k_split_epilogue<GEMM_EPI_QKV, SPLIT, KV>), grid, dim3(128), 0, st, d_rows, ep.part,
                         ep.part_stride, N, S, ep);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

// Tile rows for a row bound and output width (bf16).  Measured on MI355X over
// the projection shapes at 32..512 rows: the smallest tiles win while they
// keep the block count moderate (more, shorter blocks balance the CUs
// better); wide outputs with many rows take 64-row tiles, and the widest
// (the lm head) 128-row ones.  The tile shape does not change any result:
// every output still accumulates K in the same order.
int gemm_tile_rows(int dtype, int rows_ub, int N) {
  if (dtype != 1) return 16;
  if (rows_ub > 1024) return 256;
  // the lm head (very wide output) at 256 and 512 rows: 256 x 256 tiles,
  // 11-15 % faster there than 128 x 128 (slower at 384 and below 256 rows)
  if (N >= 65536 && rows_ub >= 256 && rows_ub % 256 == 0) return 256;
  if (rows_ub <= 16) return 16;
  const int64_t ct = (N + 127) / 128;
  const int64_t c32 = ct * ((rows_ub + 31) / 32), c64 = ct * ((rows_ub + 63) / 64);
  if (c64 > 2048) return 128;
  if (c32 > 2048 || (rows_ub > 128 && c32 > 600)) return 64;
  return 32;
}

// Tiles of 256 rows are 256 x 256 (64 x 128 per wave: twice the MFMA work per
// LDS fragment, which only pays with many blocks).  32-row tiles take 64
// columns where that measured faster in the rollout (1.5B and 7B group steps,
// ms per row bucket):
// * wide outputs (gate/up) at 33-64 rows when 128-column tiles leave fewer
//   than two blocks per CU (1.5B: 280 blocks -> 560, 644 -> 571 ms; 7B's
//   592 blocks measured slower at 1,184);
// * narrow outputs at 17-64 rows, and at 65-128 rows those with K <= 2N (QKV,
//   O), while the 64-column tiles still number fewer than the engine's
//   no-split threshold: the same block count then needs half the split-K
//   factor and the split reduction reads half the partials (1.5B at 64 rows:
//   QKV + O + down 1096 -> 993 ms; at 128 rows QKV + O 702 -> 643 ms).  7B's
//   QKV at 128 rows would cross the threshold and run unsplit, 1.6x slower;
// * the unsplit QKV (N > K) at 512 rows and more (1.5B: 512 -> 471 ms).
// All others 128 columns.  A tile shape that changes the split factor
// changes where the fp32 split sums are cut, so results move within fp32
// rounding.
int gemm_tile_cols(int dtype, int rows_ub, int N, int K) {
  const int bm = gemm_tile_rows(dtype, rows_ub, N);
  if (bm == 256) return 256;
  if (dtype == 1 && bm == 32) {
    constexpr int64_t kNoSplitBlocks = 256;   // the engine splits K below this many output tiles
    const int64_t row_tiles = (rows_ub + 31) / 32;
    if (N >= 8192)
      return rows_ub > 32 && rows_ub <= 64 && (int64_t)((N + 127) / 128) * row_tiles < 2 * kNoSplitBlocks ? 64 : 128;
    const bool splits64 = (int64_t)((N + 63) / 64) * row_tiles < kNoSplitBlocks;
    if (rows_ub <= 64 && splits64) return 64;
    if (rows_ub <= 128 && K <= 2 * N && splits64) return 64;
    if (rows_ub >= 512 && N > K) return 64;
  }
  return 128;
}

hipError_t launch_gemm(int dtype, const void* A, int lda, int64_t a_plane, const void* W, int ldw, const int* d_rows,
                       int rows_ub, int N, int K, int splits, int k_per_split, const GemmEpi& ep, hipStream_t st) {
  if (rows_ub <= 0) return hipSuccess;
  if ((splits > 1 || dtype != 1) && !ep.part) return hipErrorInvalidValue;
  if (splits > GEMM_MAX_SPLITS) return hipErrorInvalidValue;
  if ((ep.mode == GEMM_EPI_SWIGLU || ep.mode == GEMM_EPI_QKV) && N % 32) return hipErrorInvalidValue;
  if (ep.mode == GEMM_EPI_QKV && (ep.hd % 32 || 128 % ep.hd)) return hipErrorInvalidValue;
  hipError_t e;
  if (dtype == 1) {
    if (K % BK_MAX || k_per_split % BK_MAX || N % 16) return hipErrorInvalidValue;
    switch (gemm_tile_rows(dtype, rows_ub, N)) {
      case 16: e = launch_tiled<16, 128, 1, 2, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st); break;
      case 32:
        if (gemm_tile_cols(dtype, rows_ub, N, K) == 64)
          e = launch_tiled<32, 64, 1, 2, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st);
        else
          e = launch_tiled<32, 128, 1, 4, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st);
        break;
      case 64: e = launch_tiled<64, 128, 2, 4, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st); break;
      case 128: e = launch_tiled<128, 128, 4, 4, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st); break;
      default: e = launch_tiled<256, 256, 4, 8, 1>(A, lda, a_plane, W, ldw, d_rows, rows_ub, N, K, splits, k_per_split, ep, st); break;
    }
    if (e != hipSuccess || splits == 1) return e;
    return launch_split_epilogue<1, bf16_t>(d_rows, rows_ub, N, splits, ep, st);
  }
  // fp32: whole-K product into the partial buffer, then the epilogue
  if (splits != 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_gemm_f32, dim3((N + 63) / 64, (rows_ub + 3) / 4), dim3(256), 0, st, (const float*)A, lda,
                     (const float*)W, ldw, ep.part, d_rows, N, K);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_split_epilogue<0, float>(d_rows, rows_ub, N, 1, ep, st);
}
