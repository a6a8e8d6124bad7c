// gather.hip -- embedding gather, sum-pooling, SE weighting, top-k group
// mask and linear_log for the COLD scoring path on gfx950.
//
//  user_pool   one workgroup per request: user-side groups (single-valued
//              and sum-pooled behaviour sequences, Section 3.3) are gathered
//              once per request into fp32 and broadcast to every candidate
//              row of the request later (Section 3.3, parallelism: user
//              features are shared by the ads of a query).
//  gather_se   one workgroup per tile of T rows.  Ids are read field by
//              field (the column layout of Section 3.3); each thread then
//              owns 16-byte chunks of the tile's network input, laid out so
//              that the tile's output is one contiguous, fully coalesced
//              region.  Chunks hold the gathered embedding in registers
//              while the squeeze (group mean), the two SE layers and the
//              sigmoid (Section 3.2, Eq. 2) run over the tile from LDS; the
//              chunks are then reweighted by s_g (Section 3.2), optionally
//              passed through linear_log (Eq. 3) in fp32, and rounded once
//              to the storage type.
//  group_mask  per-request mean importance of each group over the request's
//              rows, then the top-k groups (Section 3.2, feature group
//              selection); ties go to the lower group index.
#include "cold_internal.h"

namespace cold {

// last q with req_off[q] <= r, clamped to [0, Q-1]
__device__ __forceinline__ int64_t request_of_row(const int32_t *req_off, int64_t Q, int64_t r) {
  int64_t lo = 0, hi = Q;  // invariant: answer in [lo, hi)
  while (hi - lo > 1) {
    int64_t mid = (lo + hi) >> 1;
    if ((int64_t)req_off[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ float linear_log(float x) {
  if (x < -1.0f) return -logf(-x) - 1.0f;
  if (x > 1.0f) return logf(x) + 1.0f;
  return x;
}

__global__ void clear_flag_kernel(int32_t *err) { *err = 0; }

// ------------------------------------------------------------- user_pool
template <typename TS, bool HASHED>
__global__ __launch_bounds__(256) void user_pool_kernel(GatherArgs a) {
  const int64_t q = blockIdx.x;
  const int64_t Q = a.Q;
  const int d = a.d, nu = a.n_user, ns = a.n_seq, nus = nu + ns;
  if (threadIdx.x == 0) {  // offsets sanity (reported in validate mode)
    bool bad = a.req_off[q + 1] < a.req_off[q];
    if (q == 0) bad |= a.req_off[0] != 0;
    if (q == Q - 1) bad |= (int64_t)a.req_off[Q] != a.R;
    for (int f = 0; f < ns; ++f) {
      int64_t lo = a.seq_off[f * Q + q], hi = a.seq_off[f * Q + q + 1];
      bad |= hi < lo || lo < 0 || hi > a.n_seq_ids;
    }
    if (bad) atomicOr(a.err, 2);
  }
  for (int it = threadIdx.x; it < nu * d; it += blockDim.x) {
    const int f = it / d, k = it - f * d;
    const int32_t row = resolve_row<HASHED>(a.user_ids, (int64_t)f * Q + q, f, a.table_rows[f],
                                            a.table_magic[f], a.err);
    const TS *tab = static_cast<const TS *>(a.tables[f]);
    a.U[(q * nus + f) * d + k] = row >= 0 ? Elem<TS>::to_f32(tab[(int64_t)row * d + k]) : 0.0f;
    if (k == 0) a.urow[q * nu + f] = row;
  }
  for (int it = threadIdx.x; it < ns * d; it += blockDim.x) {
    const int f = it / d, k = it - f * d, g = nu + f;
    int64_t lo = a.seq_off[f * Q + q], hi = a.seq_off[f * Q + q + 1];
    lo = lo < 0 ? 0 : (lo > a.n_seq_ids ? a.n_seq_ids : lo);
    hi = hi < lo ? lo : (hi > a.n_seq_ids ? a.n_seq_ids : hi);
    const TS *tab = static_cast<const TS *>(a.tables[g]);
    float acc = 0.0f;
    for (int64_t j = lo; j < hi; ++j) {  // sum-pooling in sequence order
      const int32_t row = resolve_row<HASHED>(a.seq_ids, j, g, a.table_rows[g],
                                              a.table_magic[g], a.err);
      if (row >= 0) acc += Elem<TS>::to_f32(tab[(int64_t)row * d + k]);
    }
    a.U[(q * nus + g) * d + k] = acc;
  }
}

// ------------------------------------------------------------- gather_se
template <typename TS, int MODE, bool LL, bool HASHED>
__global__ __launch_bounds__(kGatherThreads) void gather_se_kernel(GatherArgs a) {
  constexpr int EPC = Elem<TS>::kPerChunk;  // elements per 16-byte chunk
  constexpr int CPT = kGatherChunksPerThread;
  extern __shared__ __align__(16) unsigned char smem[];

  const int M = a.M, d = a.d, H = a.H;
  const int nu = a.n_user, nus = a.n_user + a.n_seq, nax = a.n_ad + a.n_cross;
  const int T = a.rows_per_tile;
  const int CPG = d / EPC;                 // chunks per group (power of two)
  const int CPR = M * CPG;                 // chunks per row
  const int64_t R = a.R, Q = a.Q;
  const int64_t r0 = (int64_t)blockIdx.x * T;
  const int tid = threadIdx.x;

  int32_t *ridx = reinterpret_cast<int32_t *>(smem);   // [T][nax]
  int32_t *rq = ridx + T * nax;                        // [T]
  float *z = reinterpret_cast<float *>(rq + T);        // [T][M]
  float *sw = z + T * M;                               // [T][M]
  float *hid = sw + T * M;                             // [T][H]

  // ---- phase 0: request of each row; ad/cross ids -> table rows (column-wise)
  for (int t = tid; t < T; t += kGatherThreads) {
    const int64_t r = r0 + t;
    rq[t] = r < R ? (int32_t)request_of_row(a.req_off, Q, r) : 0;
  }
  for (int i = tid; i < T * nax; i += kGatherThreads) {
    const int f = i / T, t = i - f * T;
    const int64_t r = r0 + t;
    const int g = nus + f;
    int32_t row = -1;
    if (r < R) {
      const bool is_ad = f < a.n_ad;
      const void *ids = is_ad ? a.ad_ids : a.cross_ids;
      const int64_t idx = (int64_t)(is_ad ? f : f - a.n_ad) * R + r;
      if constexpr (MODE == kApplyWeights) {
        // masked-out groups are never read
        const int64_t q = request_of_row(a.req_off, Q, r);
        if (a.mask[q * M + g])
          row = resolve_row<HASHED>(ids, idx, g, a.table_rows[g], a.table_magic[g], a.err);
      } else {
        row = resolve_row<HASHED>(ids, idx, g, a.table_rows[g], a.table_magic[g], a.err);
        if (a.rows_out) a.rows_out[(int64_t)g * R + r] = row;
      }
    }
    ridx[t * nax + f] = row;
  }
  __syncthreads();
  if (MODE != kApplyWeights && a.rows_out) {
    for (int i = tid; i < T * nus; i += kGatherThreads) {
      const int f = i / T, t = i - f * T;
      const int64_t r = r0 + t;
      if (r < R) a.rows_out[(int64_t)f * R + r] = f < nu ? a.urow[(int64_t)rq[t] * nu + f] : -1;
    }
  }

  // ---- phase 1: gather chunks into registers, squeeze (mean over d)
  float v[CPT][EPC];
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int i = tid + kGatherThreads * j;
    const int t = i / CPR;
    const int c = i - t * CPR;
    const int g = c / CPG, p = c - g * CPG;
    const bool valid = t < T && r0 + t < R;
#pragma unroll
    for (int e = 0; e < EPC; ++e) v[j][e] = 0.0f;
    if (valid) {
      if (g < nus) {
        bool keep = true;
        if constexpr (MODE == kApplyWeights) keep = a.mask[(int64_t)rq[t] * M + g] != 0;
        if (keep) {
          const float4 *src = reinterpret_cast<const float4 *>(
              a.U + ((int64_t)rq[t] * nus + g) * d + p * EPC);
#pragma unroll
          for (int e4 = 0; e4 < EPC / 4; ++e4) {
            const float4 w = src[e4];
            v[j][4 * e4] = w.x; v[j][4 * e4 + 1] = w.y;
            v[j][4 * e4 + 2] = w.z; v[j][4 * e4 + 3] = w.w;
          }
        }
      } else {
        const int32_t row = ridx[t * nax + (g - nus)];
        if (row >= 0) {
          const TS *tab = static_cast<const TS *>(a.tables[g]);
          const uint4 raw = *reinterpret_cast<const uint4 *>(tab + (int64_t)row * d + p * EPC);
          Elem<TS>::unpack(raw, v[j]);
        }
      }
    }
    if constexpr (MODE != kApplyWeights) {
      float part = 0.0f;
#pragma unroll
      for (int e = 0; e < EPC; ++e) part += v[j][e];
      for (int o = 1; o < CPG; o <<= 1) part += __shfl_xor(part, o);
      if (t < T && p == 0) z[t * M + g] = valid ? part / (float)d : 0.0f;
    }
  }
  __syncthreads();

  // ---- phase 2: SE weights of the tile (Eq. 2), or stored weights x mask
  if constexpr (MODE != kApplyWeights) {
    for (int it = tid; it < T * H; it += kGatherThreads) {
      const int t = it / H, jh = it - t * H;
      float acc = a.b1[jh];
      const float *w = a.w1 + (int64_t)jh * M;
      const float *zt = z + t * M;
      for (int g = 0; g < M; ++g) acc += w[g] * zt[g];
      hid[it] = acc > 0.0f ? acc : 0.0f;
    }
    __syncthreads();
    for (int it = tid; it < T * M; it += kGatherThreads) {
      const int t = it / M, g = it - t * M;
      float acc = a.b2[g];
      const float *w = a.w2 + (int64_t)g * H;
      const float *ht = hid + t * H;
      for (int jh = 0; jh < H; ++jh) acc += w[jh] * ht[jh];
      const float sg = 1.0f / (1.0f + expf(-acc));
      sw[it] = sg;
      if (a.s_buf && r0 + t < R) a.s_buf[r0 * M + it] = sg;
    }
  } else {
    for (int it = tid; it < T * M; it += kGatherThreads) {
      const int t = it / M, g = it - t * M;
      float sg = 0.0f;
      if (r0 + t < R && a.mask[(int64_t)rq[t] * M + g]) sg = a.s_buf[r0 * M + it];
      sw[it] = sg;
    }
  }
  if constexpr (MODE == kWeightsOnly) return;
  __syncthreads();

  // ---- phase 3: reweight, linear_log, round, coalesced store
  TS *X = static_cast<TS *>(a.X);
#pragma unroll
  for (int j = 0; j < CPT; ++j) {
    const int i = tid + kGatherThreads * j;
    const int t = i / CPR;
    const int c = i - t * CPR;
    const int g = c / CPG;
    if (t < T && r0 + t < R) {
      const float sg = sw[t * M + g];
      float o[EPC];
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const float x = sg * v[j][e];
        o[e] = LL ? linear_log(x) : x;
      }
      *reinterpret_cast<uint4 *>(X + (r0 * CPR + i) * EPC) = Elem<TS>::pack(o);
    }
  }
}

// ------------------------------------------------------------- group_mask
// partial[q][p][g]: sum of s over the p-th slice of request q's rows.
__global__ __launch_bounds__(256) void mask_partial_kernel(const float *s_buf, const int32_t *req_off,
                                                           int64_t R, int32_t M, int32_t P,
                                                           float *partial) {
  const int64_t q = blockIdx.y;
  const int p = blockIdx.x;
  int64_t lo = req_off[q], hi = req_off[q + 1];
  lo = lo < 0 ? 0 : (lo > R ? R : lo);
  hi = hi < lo ? lo : (hi > R ? R : hi);
  const int64_t n = hi - lo, per = (n + P - 1) / P;
  const int64_t a = lo + p * per, b = (a + per < hi) ? a + per : hi;
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    float acc = 0.0f;
    for (int64_t r = a; r < b; ++r) acc += s_buf[r * M + g];
    partial[(q * P + p) * M + g] = acc;
  }
}

__global__ __launch_bounds__(256) void mask_select_kernel(const float *partial, const int32_t *req_off,
                                                          int64_t R, int32_t M, int32_t P, int32_t k,
                                                          uint8_t *mask, uint8_t *mask_out) {
  extern __shared__ float imp[];  // [M]
  const int64_t q = blockIdx.x;
  int64_t lo = req_off[q], hi = req_off[q + 1];
  lo = lo < 0 ? 0 : (lo > R ? R : lo);
  hi = hi < lo ? lo : (hi > R ? R : hi);
  const float n = (float)(hi - lo);
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    float acc = 0.0f;
    for (int p = 0; p < P; ++p) acc += partial[(q * P + p) * M + g];
    imp[g] = n > 0.0f ? acc / n : 0.0f;
  }
  __syncthreads();
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    const float ig = imp[g];
    int rank = 0;
    for (int o = 0; o < M; ++o) {
      const float io = imp[o];
      rank += (io > ig || (io == ig && o < g)) ? 1 : 0;
    }
    const uint8_t keep = rank < k ? 1 : 0;
    mask[q * M + g] = keep;
    if (mask_out) mask_out[q * M + g] = keep;
  }
}

// ------------------------------------------------------------- launchers
template <typename TS>
static hipError_t user_pool_t(bool hashed, const GatherArgs &a, hipStream_t s) {
  if (hashed) hipLaunchKernelGGL((user_pool_kernel<TS, true>), dim3(a.Q), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((user_pool_kernel<TS, false>), dim3(a.Q), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_user_pool(int dtype, bool hashed, const GatherArgs &a, hipStream_t s) {
  if (a.Q <= 0) return hipSuccess;
  switch (dtype) {
    case kF32: return user_pool_t<float>(hashed, a, s);
    case kBF16: return user_pool_t<__bf16>(hashed, a, s);
    default: return user_pool_t<_Float16>(hashed, a, s);
  }
}

template <typename TS, int MODE, bool LL>
static hipError_t gather_se_t(bool hashed, const GatherArgs &a, hipStream_t s) {
  const int nax = a.n_ad + a.n_cross;
  const int T = a.rows_per_tile;
  const size_t shmem = sizeof(int32_t) * (size_t)(T * nax + T) +
                       sizeof(float) * (size_t)(2 * T * a.M + T * a.H);
  const dim3 grid((unsigned)((a.R + T - 1) / T));
  if (hashed)
    hipLaunchKernelGGL((gather_se_kernel<TS, MODE, LL, true>), grid, dim3(kGatherThreads), shmem, s, a);
  else
    hipLaunchKernelGGL((gather_se_kernel<TS, MODE, LL, false>), grid, dim3(kGatherThreads), shmem, s, a);
  return hipGetLastError();
}

template <typename TS>
static hipError_t gather_se_dt(int mode, bool ll, bool hashed, const GatherArgs &a, hipStream_t s) {
  if (mode == kWeightsOnly) return gather_se_t<TS, kWeightsOnly, false>(hashed, a, s);
  if (mode == kApplyWeights)
    return ll ? gather_se_t<TS, kApplyWeights, true>(hashed, a, s)
              : gather_se_t<TS, kApplyWeights, false>(hashed, a, s);
  return ll ? gather_se_t<TS, kFull, true>(hashed, a, s) : gather_se_t<TS, kFull, false>(hashed, a, s);
}

hipError_t launch_gather_se(int dtype, int mode, bool linear_log, bool hashed, const GatherArgs &a,
                            hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  switch (dtype) {
    case kF32: return gather_se_dt<float>(mode, linear_log, hashed, a, s);
    case kBF16: return gather_se_dt<__bf16>(mode, linear_log, hashed, a, s);
    default: return gather_se_dt<_Float16>(mode, linear_log, hashed, a, s);
  }
}

hipError_t launch_group_mask(const float *s_buf, const int32_t *req_off, int64_t Q, int64_t R,
                             int32_t M, int32_t k, float *partial, int32_t n_parts, uint8_t *mask,
                             uint8_t *mask_out, hipStream_t s) {
  if (Q <= 0) return hipSuccess;
  hipLaunchKernelGGL(mask_partial_kernel, dim3(n_parts, (unsigned)Q), dim3(256), 0, s, s_buf,
                     req_off, R, M, n_parts, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mask_select_kernel, dim3((unsigned)Q), dim3(256), sizeof(float) * M, s,
                     partial, req_off, R, M, n_parts, k, mask, mask_out);
  return hipGetLastError();
}

hipError_t launch_clear_flag(int32_t *err, hipStream_t s) {
  hipLaunchKernelGGL(clear_flag_kernel, dim3(1), dim3(1), 0, s, err);
  return hipGetLastError();
}

}  // namespace cold
