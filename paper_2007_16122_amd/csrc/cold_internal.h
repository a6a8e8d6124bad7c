// cold_internal.h -- device helpers and kernel launchers shared by the HIP
// sources of libcold.so (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cold {

enum Dtype { kF32 = 0, kBF16 = 1, kF16 = 2 };

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

// --------------------------------------------------------------- storage types
// Element conversions between a 16-byte chunk of storage and fp32 registers.
template <typename TS> struct Elem;

template <> struct Elem<float> {
  static constexpr int kPerChunk = 4;
  __device__ static inline void unpack(const uint4 &u, float *v) {
    v[0] = __uint_as_float(u.x); v[1] = __uint_as_float(u.y);
    v[2] = __uint_as_float(u.z); v[3] = __uint_as_float(u.w);
  }
  __device__ static inline uint4 pack(const float *v) {
    return make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]),
                      __float_as_uint(v[2]), __float_as_uint(v[3]));
  }
  __device__ static inline float to_f32(float x) { return x; }
  __device__ static inline float from_f32(float x) { return x; }
};

template <> struct Elem<__bf16> {
  static constexpr int kPerChunk = 8;
  __device__ static inline void unpack(const uint4 &u, float *v) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static inline uint16_t bits(float x) {
    __bf16 b = static_cast<__bf16>(x);  // round to nearest even
    return __builtin_bit_cast(uint16_t, b);
  }
  // pairs rounded by one vector conversion each (v_cvt_pk_bf16_f32), the same
  // round-to-nearest-even as bits()
  __device__ static inline uint4 pack(const float *v) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){v[2 * i], v[2 * i + 1]}, b2));
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static inline float to_f32(__bf16 x) { return static_cast<float>(x); }
  __device__ static inline __bf16 from_f32(float x) { return static_cast<__bf16>(x); }
};

template <> struct Elem<_Float16> {
  static constexpr int kPerChunk = 8;
  __device__ static inline void unpack(const uint4 &u, float *v) {
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = static_cast<float>(__builtin_bit_cast(_Float16, (uint16_t)(w[i] & 0xFFFFu)));
      v[2 * i + 1] = static_cast<float>(__builtin_bit_cast(_Float16, (uint16_t)(w[i] >> 16)));
    }
  }
  __device__ static inline uint16_t bits(float x) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));  // RNE, overflow -> inf
  }
  __device__ static inline uint4 pack(const float *v) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){v[2 * i], v[2 * i + 1]}, h2));
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
  __device__ static inline float to_f32(_Float16 x) { return static_cast<float>(x); }
  __device__ static inline _Float16 from_f32(float x) { return static_cast<_Float16>(x); }
};

// ------------------------------------------------------------ waits
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// wait until at most N of this wave's vector memory operations are in flight
// and all of its LDS operations have returned (s_waitcnt: vmcnt low bits
// [3:0], expcnt [6:4] left at its maximum, lgkmcnt [11:8] = 0, vmcnt high
// bits [15:14])
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// ------------------------------------------------------------ id resolution
// SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// h mod n for n < 2^31 with magic = floor((2^64 - 1) / n): the Barrett
// estimate q = mulhi(h, magic) is at most two below the true quotient, so at
// most two corrections give the exact remainder.
__device__ __forceinline__ uint32_t mod_barrett(uint64_t h, uint64_t n, uint64_t magic) {
  uint64_t q = __umul64hi(h, magic);
  uint64_t r = h - q * n;
  if (r >= n) r -= n;
  if (r >= n) r -= n;
  return (uint32_t)r;
}

// Table row of an id of feature group g, or -1 (and an error bit) for a
// direct id outside [0, rows).
template <bool HASHED>
__device__ __forceinline__ int32_t resolve_row(const void *ids, int64_t i, int g, int64_t rows,
                                               uint64_t magic, int32_t *err) {
  if constexpr (HASHED) {
    const uint64_t raw = static_cast<const uint64_t *>(ids)[i];
    const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
    return (int32_t)mod_barrett(mix64(raw ^ salt), (uint64_t)rows, magic);
  } else {
    const int32_t id = static_cast<const int32_t *>(ids)[i];
    if (id < 0 || (int64_t)id >= rows) {
      atomicOr(err, 1);
      return -1;
    }
    return id;
  }
}

// ------------------------------------------------------------ kernel params
// floor(n / d) for 0 <= n < 2^16 and 1 <= d < 2^16, from m = div_magic(d):
// with m = ceil(2^32 / d), n m / 2^32 exceeds n / d by less than n / 2^32,
// which is below 1 / d while n d < 2^32, so the floor is exact; d = 1 is m = 0
__host__ __device__ inline uint32_t div_magic(uint32_t d) {
  return d <= 1 ? 0u : (uint32_t)(0xFFFFFFFFull / d + 1);
}
__device__ __forceinline__ int fast_div(int n, uint32_t m) {
  return m ? (int)__umulhi((uint32_t)n, m) : n;
}

struct GatherArgs {
  int32_t M, n_user, n_seq, n_ad, n_cross, d, H;
  int32_t Mp, Hp;                 // M and H rounded up to multiples of 4 (LDS row strides)
  uint32_t mg_tw, mg_h, mg_m, mg_ns, mg_sd4;   // div_magic of rows_per_tile, H, M, n_seq, n_seq*d/4
  int32_t rows_per_tile;          // rows per wave (set by the launcher)
  int32_t wave_lds_bytes;         // LDS per wave (set by the launcher)
  int32_t se_lds_bytes;           // LDS for SE parameters, 0 if read from global
  int32_t se_in_lds;
  int32_t meta_lds_bytes;         // LDS for per-group table metadata
  int32_t req_lds_bytes;          // LDS for the request offsets, 0 if searched in global
  int32_t users_in_lds;           // user rows staged in LDS by the gather (no pooling pass)
  int32_t urow_lds_bytes;         // LDS for their resolved rows
  int32_t uval_lds_bytes;         // LDS for their values (storage type)
  int64_t R, Q, n_seq_ids;
  const int32_t *req_off;         // [Q+1]
  const void *user_ids;           // [n_user][Q]
  const void *ad_ids;             // [n_ad][R]
  const void *cross_ids;          // [n_cross][R]
  const int32_t *seq_off;         // [n_seq*Q+1]
  const void *seq_ids;            // [n_seq_ids]
  const void *const *tables;      // device [M]
  const int64_t *table_rows;      // device [M]
  const uint64_t *table_magic;    // device [M]
  const int32_t *cross_pairs;     // device [n_cross][2] (user field, ad field) or null
  const float *w1, *b1, *w2, *b2; // SE parameters
  const float *w1t, *w2t;         // W1 as [M][H], W2 as [H][M] (read when they are not in LDS)
  const float *w1f, *w2f;         // W1, W2 in gather_full's operand order, or null
  float *U;                       // [Q][n_user+n_seq][d] pooled user side
  float *zU;                      // [Q][n_user+n_seq] squeeze of the user groups
  void *Uh;                       // [Q][n_user][d] single-valued user rows, storage type
  int32_t *urow;                  // [Q][max(n_user,1)] resolved user rows
  void *X;                        // [R][M*d] network input
  float *s_buf;                   // [R][M] SE weights (written, or read in apply mode)
  float *z_out;                   // [R][M] squeeze (kSqueezeRaw)
  const uint8_t *mask;            // [Q][M] kept groups (apply mode)
  int32_t *rows_out;              // [M][R] or null
  int32_t *err;                   // error bits
};

// kFull: SE and reweighting in one pass; kWeightsOnly: SE weights to s_buf;
// kApplyWeights: reweight with s_buf (groups outside `mask`, when given,
// read nothing and get weight 0); kRawOut: the concatenated embedding in
// fp32 to X, for an SE computed elsewhere
// kSqueezeRaw: the squeeze to z_out [R][M] and the gathered rows, exact in the
// storage type, to X, for se_rows and apply_weights (models without sequences)
enum GatherMode { kFull = 0, kWeightsOnly = 1, kApplyWeights = 2, kRawOut = 3, kSqueezeRaw = 4 };

// launchers (return hipError_t of the launch)
bool user_pool_needed(int dtype, const GatherArgs &a);
hipError_t launch_user_pool(int dtype, bool hashed, const GatherArgs &a, hipStream_t s);
// the register-resident kFull gather (M <= 48, H <= 16, 32-byte group rows,
// no sequences; needs the packed SE operands, and the pooling pass where
// user_pool_needed says so)
constexpr int kSeFullFloats = 4 * 64 * 4;   // floats of each packed operand
bool gather_full_shape(int32_t M, int32_t H, int32_t row_bytes, int32_t n_seq);
bool gather_full_supported(int dtype, const GatherArgs &a);
hipError_t launch_gather_full(int dtype, bool linear_log, bool hashed, const GatherArgs &a,
                              hipStream_t s);
hipError_t launch_pack_se_full(const float *w1, const float *w2, int32_t M, int32_t H, float *w1f,
                               float *w2f, hipStream_t s);
hipError_t launch_gather_se(int dtype, int mode, bool linear_log, bool hashed,
                            const GatherArgs &a, hipStream_t s);
hipError_t launch_group_mask(const float *s_buf, const int32_t *req_off, int64_t Q, int64_t R,
                             int32_t M, int32_t k, float *partial, int32_t n_parts,
                             uint8_t *mask, uint8_t *mask_out, hipStream_t s);
hipError_t launch_clear_flag(int32_t *err, hipStream_t s);
// compute units of the current device (cached per device; 0 on error)
int device_cus();
// SE weights of every row from its squeeze (Eq. 2 read as squeeze ->
// FC -> ReLU -> FC -> sigmoid): s [R][M] from z [R][M] on the fp32 matrix
// cores, with W1 and W2 packed by launch_pack_se_rows; M <= 256, H <= 64
// (tile_part, when not null: [ceil(R / 16)][M] sums of s over each 16-row tile)
hipError_t launch_se_rows(const float *z, float *s_out, int64_t R, int32_t M, int32_t H,
                          const float *w1p, const float *b1, const float *w2p, const float *b2,
                          float *tile_part, hipStream_t s);
// the top-k mask of every request from s [R][M] and se_rows' tile sums;
// kept (when not null, M <= 256): [Q][min(k, M)] the kept groups in group order
hipError_t launch_group_mask_tiles(const float *s_buf, const float *tile_part,
                                   const int32_t *req_off, int64_t Q, int64_t R, int32_t M,
                                   int32_t k, uint8_t *mask, uint8_t *mask_out, int32_t *kept,
                                   hipStream_t s);

// floats of the two packed SE operands (0 when M or H is beyond the kernel)
void se_rows_packed_floats(int32_t M, int32_t H, size_t *n1, size_t *n2);
// W1 [H][M] and W2 [M][H] into the row-wise SE kernel's operand order
hipError_t launch_pack_se_rows(const float *w1, const float *w2, int32_t M, int32_t H, float *w1p,
                               float *w2p, hipStream_t s);
// X [R][M*d] in place: the gathered rows (storage type) times s [R][M] and
// the request's group mask [Q][M] (NULL: all kept), linear_log when ll,
// rounded once to the storage type
hipError_t launch_apply_weights(int dtype, bool ll, void *X, const float *s_buf,
                                const uint8_t *mask, const int32_t *req_off, int64_t Q, int64_t R,
                                int32_t M, int32_t d, hipStream_t s);
// dst[c][r] = src[r][c] for a [rows][cols] fp32 matrix
hipError_t launch_transpose_f32(const float *src, float *dst, int32_t rows, int32_t cols,
                                hipStream_t s);

hipError_t launch_dense_relu(int dtype, const void *x, const void *w, const float *b, void *y,
                             int64_t R, int32_t N, int32_t K, hipStream_t s);
// One row tile of a layer whose requests each have their own weights: rows
// [r0, r0 + n) of request q
struct RowTile {
  int64_t r0;
  int32_t n, q;
};
// entries of the row-tile table for R rows in Q requests (any tile height)
inline int64_t row_tile_capacity(int64_t R, int64_t Q) { return (R + 63) / 64 + Q + 1; }
// Row tiles of height BR over requests: the bound on their count (request q
// of n_q rows takes ceil(n_q / BR) <= (n_q + BR - 1) / BR tiles; exact for
// one request, so a one-request batch has no idle workgroups).
inline int64_t row_tiles_bound(int64_t R, int64_t Q, int BR) { return (R + Q * (BR - 1)) / BR; }

// The table of those tiles, by one workgroup of NT threads: request q's rows
// [lo, hi) (offsets clamped to [0, R]) take ceil((hi - lo) / BR) tiles, in
// request order; entries past cap are not written (cap bounds the table and
// the layer's grid whatever the offsets are). Requests in blocks of NT with
// a running start.
template <int NT>
__device__ void build_row_tiles(const int32_t *__restrict__ req_off, int64_t Q, int64_t R, int BR,
                                int64_t cap, RowTile *__restrict__ tiles,
                                int32_t *__restrict__ n_tiles, int64_t *s_scan) {
  const int tid = threadIdx.x;
  int64_t start0 = 0;
  for (int64_t base = 0; base < Q; base += NT) {
    const int64_t q = base + tid;
    int64_t lo = 0, hi = 0;
    if (q < Q) {
      lo = req_off[q];
      hi = req_off[q + 1];
      lo = lo < 0 ? 0 : (lo > R ? R : lo);
      hi = hi < lo ? lo : (hi > R ? R : hi);
    }
    const int64_t c = (hi - lo + BR - 1) / BR;
    s_scan[tid] = c;
    __syncthreads();
    for (int off = 1; off < NT; off <<= 1) {
      const int64_t v = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += v;
      __syncthreads();
    }
    const int64_t start = start0 + s_scan[tid] - c;
    for (int64_t t = 0; t < c && start + t < cap; ++t) {
      const int64_t r = lo + t * BR;
      RowTile e;
      e.r0 = r;
      e.n = (int32_t)(hi - r < BR ? hi - r : BR);
      e.q = (int32_t)q;
      tiles[start + t] = e;
    }
    start0 += s_scan[NT - 1];
    __syncthreads();   // s_scan is rewritten by the next block of requests
  }
  if (tid == 0) n_tiles[0] = (int32_t)(start0 < cap ? start0 : cap);
}

// rows of the tile launch_dense_relu_grouped uses for R rows, N outputs and K inputs
int dense_grouped_tile_rows(int64_t R, int32_t N, int32_t K);
// Y = ReLU(X W_q^T + b) where row r of X [R][K] belongs to request q(r)
// and W_q = W + q * N * K; the row tiles, which never straddle two
// requests, come from the table and count that launch_apply_compact built
// for the same R, Q, N and K.
// Same tile shapes and sum order as launch_dense_relu; bf16 and fp16 with
// K % 32 == 0 and N % 8 == 0.
bool dense_grouped_supported(int dtype, int32_t N, int32_t K);
// Xc [R][kp*d]: the kp kept groups of each row's request (kept [Q][kp]) taken
// from the gathered rows Xraw [R][M*d], times s [R][M], linear_log when ll,
// rounded once to the storage type. The same launch writes Wc [Q][N][kp*d],
// every request's columns of the first layer's weights W [N][M*d] for its
// kept groups, and lays out the row tiles of launch_dense_relu_grouped for
// these R rows (tiles [row_tile_capacity], n_tiles [1]).
hipError_t launch_apply_compact(int dtype, bool ll, const void *Xraw, void *Xc, const float *s_buf,
                                const int32_t *kept, const int32_t *req_off, int64_t Q, int64_t R,
                                int32_t M, int32_t kp, int32_t d, const void *W, int32_t N,
                                void *Wc, RowTile *tiles, int32_t *n_tiles, hipStream_t s);
hipError_t launch_dense_relu_grouped(int dtype, const void *x, const void *w, const float *b,
                                     void *y, int64_t R, int64_t Q, int32_t N, int32_t K,
                                     RowTile *tiles, int32_t *n_tiles, hipStream_t s);
bool tail_supported(int dtype, int K0, int N1, int N2, int n_out);
// the fused tail reads its two hidden layers' weights fragment-major
// (mlp.hip, frag_offset): [N][K] row-major -> that order (N % 16 == 0, K % 32 == 0)
hipError_t launch_pack_frag(const void *src, void *dst, int64_t N, int32_t K, hipStream_t s);
hipError_t launch_mlp_tail(int dtype, const void *a, const void *w1, const float *b1,
                           const void *w2, const float *b2, const void *wh, const float *bh,
                           int32_t n_out, float *scores, int64_t R, hipStream_t s);
// the last separate hidden layer (N = 256, the tail's input) and the fused
// tail in one kernel; hipErrorNotSupported unless N == 256, K % 64 == 0 and
// the model is in half precision
bool dense_tail_supported(int dtype, int64_t R, int32_t N, int32_t K);
hipError_t launch_dense_tail(int dtype, const void *x, const void *w, const float *b, int32_t N,
                             int32_t K, const void *w1, const float *b1, const void *w2,
                             const float *b2, const void *wh, const float *bh, int32_t n_out,
                             float *scores, int64_t R, hipStream_t s);
hipError_t launch_dense_f32(const float *x, const float *w, const float *b, float *y, int64_t R,
                            int32_t N, int32_t K, int act, hipStream_t s);
hipError_t launch_topn(const float *scores, const float *bids, const int32_t *req_off, int64_t Q,
                       int64_t R, int32_t n_top, int32_t *top_rows, float *top_ecpm, hipStream_t s);
hipError_t launch_head(int dtype, const void *a, const void *w, const float *b, float *scores,
                       int64_t R, int32_t K, int32_t n_out, hipStream_t s);

constexpr int kGatherThreads = 256;
constexpr int kGatherMaxChunksPerRow = 1024;  // 64 lanes x 16 chunks
constexpr int kGatherMaxIdsPerLane = 8;       // rows per wave x (ad + cross fields) <= 512
constexpr int kMaskParts = 256;   // row parts per request in the importance reduction
constexpr int kGatherMaxReqLds = 1024;        // request offsets held in LDS up to this count
constexpr int kGatherMaxUserValLds = 4096;    // user row bytes the gather stages in LDS itself

}  // namespace cold
