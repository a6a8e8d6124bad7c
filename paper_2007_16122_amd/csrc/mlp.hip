// mlp.hip -- the fully connected network of the COLD model (Section 4.1:
// D_in x 1024 x 512 x 256 x 128 x 64 x 2) on gfx950.
//
//  dense_relu_mfma  Y = ReLU(X W^T + b) for bf16/fp16 X, W with fp32
//                   accumulation on the matrix cores
//                   (v_mfma_f32_16x16x32_{bf16,f16}), one rounding of the
//                   output to the storage type.  256 threads = 4 waves per
//                   128-row tile; W plays the MFMA A operand (output features
//                   on the rows) and X the B operand, so each lane ends with
//                   4 consecutive output features of one row (one 8-byte
//                   store).  Tiles of both operands go through LDS, double
//                   buffered, one barrier per 32-deep K step; rows are
//                   padded by 16 bytes so the 16-byte fragment reads of a
//                   wave hit distinct LDS banks.  Tiles are numbered so that
//                   the workgroups sharing one row block of X run on the same
//                   XCD (workgroup i is dispatched to XCD i mod 8) and reuse
//                   it from that XCD's L2.
//  dense_relu_f32   the same layer in fp32 FMA (the fp32 model).
//  head             last layer (n_out = 1 or 2) in fp32 plus sigmoid or
//                   two-way softmax; writes the CTR.
#include "cold_internal.h"

namespace cold {

constexpr int kBM = 128;   // rows of X per tile
constexpr int kBK = 32;    // K per step (one MFMA depth)
constexpr int kPad = 8;    // elements of row padding in LDS
constexpr int kLdsRow = kBK + kPad;

template <typename TS> struct Mfma;
template <> struct Mfma<__bf16> {
  typedef bf16x8 frag;
  __device__ static inline f32x4 mac(const frag &a, const frag &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<_Float16> {
  typedef f16x8 frag;
  __device__ static inline f32x4 mac(const frag &a, const frag &b, const f32x4 &c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  }
};

// XCD-aware tile order: workgroup b runs on XCD b % 8; give XCD x the
// contiguous tile range [start_x, start_x + count_x).
__device__ __forceinline__ int xcd_tile(int b, int total) {
  const int x = b & 7, slot = b >> 3;
  const int base = total >> 3, extra = total & 7;
  const int start = x * base + (x < extra ? x : extra);
  return start + slot;
}

template <typename TS, int BN>
__global__ __launch_bounds__(256) void dense_relu_mfma_kernel(const TS *__restrict__ X,
                                                              const TS *__restrict__ W,
                                                              const float *__restrict__ bias,
                                                              TS *__restrict__ Y, int64_t R, int N,
                                                              int K, int tiles_n, int tiles_total) {
  typedef typename Mfma<TS>::frag frag;
  constexpr int NI = BN / 2 / 16;          // 16-wide output-feature blocks per wave
  constexpr int RJ = 4;                    // 16-wide row blocks per wave (64 rows)
  constexpr int A_CHUNKS = BN * kBK / 8;   // 16-byte chunks of the W tile
  constexpr int B_CHUNKS = kBM * kBK / 8;
  constexpr int A_PER_T = A_CHUNKS / 256, B_PER_T = B_CHUNKS / 256;
  static_assert(A_CHUNKS % 256 == 0 && B_CHUNKS % 256 == 0, "tile/thread mismatch");

  __shared__ __align__(16) TS sA[2][BN * kLdsRow];
  __shared__ __align__(16) TS sB[2][kBM * kLdsRow];

  const int tile = xcd_tile(blockIdx.x, tiles_total);
  const int tr = tile / tiles_n, tn = tile - tr * tiles_n;
  const int64_t r0 = (int64_t)tr * kBM;
  const int n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wr = wave >> 1;

  uint4 ra[A_PER_T], rb[B_PER_T];
  auto load_global = [&](int k0) {
#pragma unroll
    for (int u = 0; u < A_PER_T; ++u) {
      const int c = tid + 256 * u, row = c >> 2, kc = (c & 3) * 8;
      const int n = n0 + row, k = k0 + kc;
      ra[u] = (n < N && k < K) ? *reinterpret_cast<const uint4 *>(W + (int64_t)n * K + k)
                               : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < B_PER_T; ++u) {
      const int c = tid + 256 * u, row = c >> 2, kc = (c & 3) * 8;
      const int64_t r = r0 + row;
      const int k = k0 + kc;
      rb[u] = (r < R && k < K) ? *reinterpret_cast<const uint4 *>(X + r * K + k)
                               : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_lds = [&](int buf) {
#pragma unroll
    for (int u = 0; u < A_PER_T; ++u) {
      const int c = tid + 256 * u, row = c >> 2, kc = (c & 3) * 8;
      *reinterpret_cast<uint4 *>(&sA[buf][row * kLdsRow + kc]) = ra[u];
    }
#pragma unroll
    for (int u = 0; u < B_PER_T; ++u) {
      const int c = tid + 256 * u, row = c >> 2, kc = (c & 3) * 8;
      *reinterpret_cast<uint4 *>(&sB[buf][row * kLdsRow + kc]) = rb[u];
    }
  };

  f32x4 acc[NI][RJ];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < RJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ksteps = (K + kBK - 1) / kBK;
  load_global(0);
  store_lds(0);
  __syncthreads();
  const int frow = lane & 15, fk = (lane >> 4) * 8;
  for (int ks = 0; ks < ksteps; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < ksteps) load_global((ks + 1) * kBK);
    frag fa[NI], fb[RJ];
#pragma unroll
    for (int i = 0; i < NI; ++i)
      fa[i] = *reinterpret_cast<const frag *>(&sA[buf][(wn * (BN / 2) + i * 16 + frow) * kLdsRow + fk]);
#pragma unroll
    for (int j = 0; j < RJ; ++j)
      fb[j] = *reinterpret_cast<const frag *>(&sB[buf][(wr * 64 + j * 16 + frow) * kLdsRow + fk]);
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < RJ; ++j) acc[i][j] = Mfma<TS>::mac(fa[i], fb[j], acc[i][j]);
    if (ks + 1 < ksteps) store_lds(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds D[4*(lane/16) + e][lane % 16], e = 0..3, of each block
  const int dn = (lane >> 4) * 4, dr = lane & 15;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int n = n0 + wn * (BN / 2) + i * 16 + dn;
    if (n >= N) continue;
    float bv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) bv[e] = (n + e < N) ? bias[n + e] : 0.0f;
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
      const int64_t r = r0 + wr * 64 + j * 16 + dr;
      if (r >= R) continue;
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = acc[i][j][e] + bv[e];
        o[e] = t > 0.0f ? t : 0.0f;
      }
      if (n + 3 < N) {
        uint2 packed;
        packed.x = (uint32_t)Elem<TS>::bits(o[0]) | ((uint32_t)Elem<TS>::bits(o[1]) << 16);
        packed.y = (uint32_t)Elem<TS>::bits(o[2]) | ((uint32_t)Elem<TS>::bits(o[3]) << 16);
        *reinterpret_cast<uint2 *>(Y + r * N + n) = packed;
      } else {
        for (int e = 0; e < 4 && n + e < N; ++e) Y[r * N + n + e] = Elem<TS>::from_f32(o[e]);
      }
    }
  }
}

// fp32 layer: 64 x 64 output tile, 4 x 4 per thread, K in steps of 16.
__global__ __launch_bounds__(256) void dense_relu_f32_kernel(const float *__restrict__ X,
                                                             const float *__restrict__ W,
                                                             const float *__restrict__ bias,
                                                             float *__restrict__ Y, int64_t R,
                                                             int N, int K, int relu) {
  __shared__ float sx[16][64 + 1];
  __shared__ float sw[16][64 + 1];
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  const int tr = tid >> 4, tn = tid & 15;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int i = tid; i < 64 * 16; i += 256) {
      const int row = i >> 4, kk = i & 15;
      const int64_t r = r0 + row;
      const int n = n0 + row, k = k0 + kk;
      sx[kk][row] = (r < R && k < K) ? X[r * K + k] : 0.0f;
      sw[kk][row] = (n < N && k < K) ? W[(int64_t)n * K + k] : 0.0f;
    }
    __syncthreads();
    for (int kk = 0; kk < 16; ++kk) {
      float xv[4], wv[4];
      for (int a = 0; a < 4; ++a) xv[a] = sx[kk][tr * 4 + a];
      for (int b = 0; b < 4; ++b) wv[b] = sw[kk][tn * 4 + b];
      for (int a = 0; a < 4; ++a)
        for (int b = 0; b < 4; ++b) acc[a][b] += xv[a] * wv[b];
    }
    __syncthreads();
  }
  for (int a = 0; a < 4; ++a) {
    const int64_t r = r0 + tr * 4 + a;
    if (r >= R) continue;
    for (int b = 0; b < 4; ++b) {
      const int n = n0 + tn * 4 + b;
      if (n >= N) continue;
      const float t = acc[a][b] + bias[n];
      Y[r * N + n] = (relu && t < 0.0f) ? 0.0f : t;
    }
  }
}

// last layer + sigmoid (n_out = 1) or softmax (n_out = 2, CTR = class 1)
template <typename TS>
__global__ __launch_bounds__(256) void head_kernel(const TS *__restrict__ A, const TS *__restrict__ W,
                                                   const float *__restrict__ bias,
                                                   float *__restrict__ scores, int64_t R, int K,
                                                   int n_out) {
  extern __shared__ float sw[];  // [n_out][K]
  for (int i = threadIdx.x; i < n_out * K; i += blockDim.x) sw[i] = Elem<TS>::to_f32(W[i]);
  __syncthreads();
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  const TS *a = A + r * K;
  float z0 = bias[0], z1 = n_out > 1 ? bias[1] : 0.0f;
  for (int k = 0; k < K; ++k) {
    const float x = Elem<TS>::to_f32(a[k]);
    z0 += sw[k] * x;
    if (n_out > 1) z1 += sw[K + k] * x;
  }
  scores[r] = n_out == 1 ? 1.0f / (1.0f + expf(-z0)) : 1.0f / (1.0f + expf(z0 - z1));
}

// ------------------------------------------------------------- launchers
template <typename TS, int BN>
static hipError_t dense_mfma_t(const void *x, const void *w, const float *b, void *y, int64_t R,
                               int N, int K, hipStream_t s) {
  const int tiles_n = (N + BN - 1) / BN;
  const int64_t tiles_r = (R + kBM - 1) / kBM;
  const int64_t total = tiles_r * tiles_n;
  if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dense_relu_mfma_kernel<TS, BN>), dim3((unsigned)total), dim3(256), 0, s,
                     static_cast<const TS *>(x), static_cast<const TS *>(w), b,
                     static_cast<TS *>(y), R, N, K, tiles_n, (int)total);
  return hipGetLastError();
}

template <typename TS>
static hipError_t dense_mfma_dt(const void *x, const void *w, const float *b, void *y, int64_t R,
                                int N, int K, hipStream_t s) {
  if (N % 128 == 0) return dense_mfma_t<TS, 128>(x, w, b, y, R, N, K, s);
  return dense_mfma_t<TS, 64>(x, w, b, y, R, N, K, s);
}

hipError_t launch_dense_relu(int dtype, const void *x, const void *w, const float *b, void *y,
                             int64_t R, int32_t N, int32_t K, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (dtype == kF32) {
    const dim3 grid((unsigned)((R + 63) / 64), (unsigned)((N + 63) / 64));
    hipLaunchKernelGGL(dense_relu_f32_kernel, grid, dim3(256), 0, s, static_cast<const float *>(x),
                       static_cast<const float *>(w), b, static_cast<float *>(y), R, N, K, 1);
    return hipGetLastError();
  }
  if (dtype == kBF16) return dense_mfma_dt<__bf16>(x, w, b, y, R, N, K, s);
  return dense_mfma_dt<_Float16>(x, w, b, y, R, N, K, s);
}

hipError_t launch_head(int dtype, const void *a, const void *w, const float *b, float *scores,
                       int64_t R, int32_t K, int32_t n_out, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  const dim3 grid((unsigned)((R + 255) / 256));
  const size_t sh = sizeof(float) * (size_t)n_out * K;
  switch (dtype) {
    case kF32:
      hipLaunchKernelGGL(head_kernel<float>, grid, dim3(256), sh, s, static_cast<const float *>(a),
                         static_cast<const float *>(w), b, scores, R, K, n_out);
      break;
    case kBF16:
      hipLaunchKernelGGL(head_kernel<__bf16>, grid, dim3(256), sh, s,
                         static_cast<const __bf16 *>(a), static_cast<const __bf16 *>(w), b, scores,
                         R, K, n_out);
      break;
    default:
      hipLaunchKernelGGL(head_kernel<_Float16>, grid, dim3(256), sh, s,
                         static_cast<const _Float16 *>(a), static_cast<const _Float16 *>(w), b,
                         scores, R, K, n_out);
  }
  return hipGetLastError();
}

}  // namespace cold
