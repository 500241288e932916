// Device-side helpers shared by the rollout kernels (gfx950 / CDNA4, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define RG_WAVE 64

typedef uint16_t bf16_t;  // raw bfloat16 bit pattern
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bfloat16
__device__ __forceinline__ float bf16_to_f32(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// Round a finite fp32 value to the nearest bfloat16, ties to even.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t b = __float_as_uint(f);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (bf16_t)(b >> 16);
}

// Two fp32 values as packed bfloat16 (a in the low half), rounded to nearest
// even by v_cvt_pk_bf16_f32; equal to f32_to_bf16 on finite values.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// Storage types: the activation / KV element type is either float or bf16_t.
template <typename T> __device__ __forceinline__ float ld_f32(const T* p);
template <> __device__ __forceinline__ float ld_f32<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ld_f32<bf16_t>(const bf16_t* p) { return bf16_to_f32(*p); }
template <typename T> __device__ __forceinline__ void st_from_f32(T* p, float v);
template <> __device__ __forceinline__ void st_from_f32<float>(float* p, float v) { *p = v; }
template <> __device__ __forceinline__ void st_from_f32<bf16_t>(bf16_t* p, float v) { *p = f32_to_bf16(v); }

// ---------------------------------------------------------------- activations
// Activation operand of a matrix product.  fp32 models: one fp32 plane.
// bf16 models: two bf16 planes, hi = bf16(v) and lo = bf16(v - hi) (v - hi is
// exact in fp32), so hi + lo carries v to within 2^-17 relative and the MFMA
// product W*hi + W*lo keeps the activation's precision.
struct ActOut {
  void* base;
  int64_t plane;  // elements between the hi and lo planes (bf16 models)
};

template <int SPLIT> __device__ __forceinline__ void act_store(ActOut o, int64_t i, float v);
template <> __device__ __forceinline__ void act_store<0>(ActOut o, int64_t i, float v) { ((float*)o.base)[i] = v; }
template <> __device__ __forceinline__ void act_store<1>(ActOut o, int64_t i, float v) {
  const bf16_t h = f32_to_bf16(v);
  bf16_t* p = (bf16_t*)o.base;
  p[i] = h;
  p[o.plane + i] = f32_to_bf16(v - bf16_to_f32(h));
}

// ---------------------------------------------------------------- Philox4x64-10
// Counter-based generator of Salmon et al. (SC'11): 4x64-bit counter, 2x64-bit
// key, ten rounds; each round takes the 128-bit products of counter words 0
// and 2 with two odd multipliers, swaps/XORs the halves with words 1 and 3 and
// the key, and the key advances by two Weyl constants between rounds.
struct rg_u64x4 { uint64_t v[4]; };

__device__ __forceinline__ void rg_mulhilo64(uint64_t a, uint64_t b, uint64_t& hi, uint64_t& lo) {
  lo = a * b;
  hi = __umul64hi(a, b);
}

__device__ __forceinline__ rg_u64x4 rg_philox4x64_10(rg_u64x4 c, uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += W0; k1 += W1; }
    uint64_t hi0, lo0, hi1, lo1;
    rg_mulhilo64(M0, c.v[0], hi0, lo0);
    rg_mulhilo64(M1, c.v[2], hi1, lo1);
    rg_u64x4 n;
    n.v[0] = hi1 ^ c.v[1] ^ k0;
    n.v[1] = lo1;
    n.v[2] = hi0 ^ c.v[3] ^ k1;
    n.v[3] = lo0;
    c = n;
  }
  return c;
}

// Sampling stream: key (seed, RG_TAG_GUMBEL), counter (v >> 3, t, s, 0); value
// j = v & 7 of a block is the (j & 1)-th 32-bit half (low first) of word j >> 1.
#define RG_TAG_GUMBEL 1ull

// 32-bit value x -> fp32 uniform (2*(x >> 9) + 1) * 2^-24, exactly, in (0, 1).
__device__ __forceinline__ float rg_uniform_from_bits(uint32_t x) {
  return (float)(2u * (x >> 9) + 1u) * 5.9604644775390625e-08f;  // 2^-24
}

// ---------------------------------------------------------------- reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, RG_WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, RG_WAVE));
  return v;
}
__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, RG_WAVE);
  return v;
}

// Block-wide sum over blockDim.x threads (a multiple of 64, <= 1024).
// `red` must hold 16 floats of shared memory.  All threads get the result.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < nw; ++i) r += red[i];
  return r;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float r = -INFINITY;
  for (int i = 0; i < nw; ++i) r = fmaxf(r, red[i]);
  return r;
}

// Exclusive prefix sum over the block (blockDim.x multiple of 64, <= 1024);
// `lds` holds 17 ints.  Returns this thread's exclusive prefix; *total gets
// the block sum.  Contains barriers: every thread must call it.
static __device__ int block_excl_scan(int v, int* lds, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds[w] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int i = 0; i < nw; ++i) { int tmp = lds[i]; lds[i] = run; run += tmp; }
    lds[16] = run;
  }
  __syncthreads();
  const int excl = lds[w] + x - v;
  *total = lds[16];
  __syncthreads();
  return excl;
}

// 1 when every G[p] >= 1 and sum(G) == N, summed in 64 bits so that no
// choice of G can wrap around to a false match.  Block-wide: every thread of
// the block calls it and gets the same answer.
static __device__ bool groups_valid(const int32_t* __restrict__ G, int P, int N) {
  __shared__ unsigned long long s_sum;
  __shared__ int s_bad;
  if (threadIdx.x == 0) { s_sum = 0; s_bad = 0; }
  __syncthreads();
  long long loc = 0;
  int bad = 0;
  for (int p = threadIdx.x; p < P; p += blockDim.x) {
    const int g = G[p];
    bad |= g < 1;
    loc += g;
  }
  if (bad) atomicOr(&s_bad, 1);
  atomicAdd(&s_sum, (unsigned long long)loc);
  __syncthreads();
  const bool ok = !s_bad && s_sum == (unsigned long long)N;
  __syncthreads();
  return ok;
}
