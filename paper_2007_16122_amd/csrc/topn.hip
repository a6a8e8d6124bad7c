// topn.hip -- per-request top-n selection by eCPM = pCTR * bid, the step
// that follows scoring in a pre-ranking system (Section 2: the pre-ranking
// model keeps the N candidates of a request with the highest eCPM; its
// footnote defines eCPM = pCTR * bid for CPC bidding).
//
// One 1024-thread workgroup per request.  Every row gets a 32-bit key, the
// IEEE-754 totalOrder rank of its fp32 eCPM (larger key = larger eCPM).  A
// four-pass radix select (8 bits per pass, histograms in LDS) finds the key
// T of the n-th best row and how many rows with key T are still needed; one
// pass in row order then collects the rows above T and the first rows equal
// to T (ties go to the lower row index), and every winner finds its place
// by counting the winners ahead of it.  Requests of up to kTopnCache rows keep their keys in LDS
// after the first pass; longer requests recompute them from global memory
// (L2) in every pass.
#include "cold.h"
#include "cold_internal.h"

namespace cold {

namespace {

constexpr int kTopnThreads = 1024;
constexpr int kTopnCache = 8192;

// totalOrder rank of an fp32 value: negative values (sign bit set) map to
// the complement of their bits, non-negative ones get the sign bit set, so
// unsigned comparison of ranks is totalOrder comparison of the values.
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}

__global__ __launch_bounds__(kTopnThreads) void topn_kernel(const float *__restrict__ scores,
                                                            const float *__restrict__ bids,
                                                            const int32_t *__restrict__ req_off,
                                                            int64_t R, int32_t n_top,
                                                            int32_t *__restrict__ top_rows,
                                                            float *__restrict__ top_ecpm) {
  __shared__ uint32_t s_keys[kTopnCache];
  __shared__ uint32_t s_hist[256];
  __shared__ uint64_t s_sel[COLD_TOPN_MAX];
  __shared__ uint64_t s_out[COLD_TOPN_MAX];
  __shared__ uint32_t s_wave_eq[kTopnThreads / 64];
  __shared__ uint32_t s_prefix, s_need, s_gt, s_eq_base;

  const int64_t q = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int64_t lo = req_off[q], hi = req_off[q + 1];
  lo = lo < 0 ? 0 : (lo > R ? R : lo);
  hi = hi < lo ? lo : (hi > R ? R : hi);
  const int64_t C = hi - lo;
  const int n = C < n_top ? (int)C : n_top;
  const bool cached = C <= kTopnCache;

  auto key_at = [&](int64_t i) -> uint32_t {   // i: row index within the request
    if (cached) return s_keys[i];
    return order_key(scores[lo + i] * bids[lo + i]);
  };

  if (n > 0) {
    if (cached)
      for (int64_t i = tid; i < C; i += kTopnThreads) s_keys[i] = order_key(scores[lo + i] * bids[lo + i]);
    if (tid == 0) { s_prefix = 0; s_need = (uint32_t)n; }
    // ---- radix select: after the pass at `shift`, s_prefix holds the top
    //      bits of T and s_need how many rows matching them are still needed
    uint32_t pmask = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) s_hist[tid] = 0;
      __syncthreads();
      const uint32_t prefix = s_prefix;
      for (int64_t i = tid; i < C; i += kTopnThreads) {
        const uint32_t u = key_at(i);
        if ((u & pmask) == prefix) atomicAdd(&s_hist[(u >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (wave == 0) {
        // lane l owns bins 255-4l .. 252-4l (best first); a prefix sum over
        // the lanes gives the count in better bins, and the first lane
        // whose bins reach `need` picks the digit
        const uint32_t need = s_need;
        uint32_t h[4], own = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) { h[e] = s_hist[255 - (4 * lane + e)]; own += h[e]; }
        uint32_t incl = own;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t t = __shfl_up(incl, o);
          if (lane >= o) incl += t;
        }
        uint32_t above = incl - own;
        int hit = -1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (hit < 0) {
            if (above + h[e] >= need) hit = e;
            else above += h[e];
          }
        }
        const uint64_t ball = __ballot(hit >= 0);
        if (hit >= 0 && lane == __ffsll((unsigned long long)ball) - 1) {
          s_prefix = prefix | ((uint32_t)(255 - (4 * lane + hit)) << shift);
          s_need = need - above;
        }
      }
      pmask |= 255u << shift;
      __syncthreads();
    }
    const uint32_t T = s_prefix;
    const uint32_t need_eq = s_need;              // rows with key T to take, >= 1
    const uint32_t n_gt = (uint32_t)n - need_eq;  // rows with key > T
    if (tid == 0) { s_gt = 0; s_eq_base = 0; }
    __syncthreads();
    // ---- collect in row order: rows above T anywhere in [0, n_gt), the
    //      first need_eq rows equal to T after them
    for (int64_t base = 0; base < C; base += kTopnThreads) {
      const int64_t i = base + tid;
      const uint32_t u = i < C ? key_at(i) : 0u;
      const bool gt = i < C && u > T, eq = i < C && u == T;
      const uint64_t sort_key = ((uint64_t)u << 32) | (uint32_t)~(uint32_t)i;
      if (gt) {
        const uint32_t pos = atomicAdd(&s_gt, 1u);
        if (pos < n_gt) s_sel[pos] = sort_key;   // exactly n_gt rows are above T
      }
      const uint64_t ball = __ballot(eq);
      const uint32_t rank_in_wave = (uint32_t)__popcll(ball & ((1ull << lane) - 1ull));
      if (lane == 0) s_wave_eq[wave] = (uint32_t)__popcll(ball);
      __syncthreads();
      uint32_t before = s_eq_base;
      for (int w = 0; w < wave; ++w) before += s_wave_eq[w];
      if (eq && before + rank_in_wave < need_eq) s_sel[n_gt + before + rank_in_wave] = sort_key;
      __syncthreads();
      if (tid == 0) {
        uint32_t tot = 0;
        for (int w = 0; w < kTopnThreads / 64; ++w) tot += s_wave_eq[w];
        s_eq_base += tot;
      }
      __syncthreads();
    }
    // ---- order the n winners, best (largest key) first: the keys are
    //      distinct, so each one's rank is the count of larger keys
    __syncthreads();
    if (tid < n) {
      const uint64_t mine = s_sel[tid];
      int rank = 0;
      for (int j = 0; j < n; ++j) rank += s_sel[j] > mine ? 1 : 0;
      s_out[rank] = mine;
    }
    __syncthreads();
  }
  for (int j = tid; j < n_top; j += kTopnThreads) {
    int32_t row = -1;
    float e = -INFINITY;
    if (j < n) {
      const uint64_t s = s_out[j];
      row = (int32_t)(lo + (int64_t)(uint32_t)~(uint32_t)s);
      e = key_value((uint32_t)(s >> 32));
    }
    top_rows[q * n_top + j] = row;
    if (top_ecpm) top_ecpm[q * n_top + j] = e;
  }
}

}  // namespace

hipError_t launch_topn(const float *scores, const float *bids, const int32_t *req_off, int64_t Q,
                       int64_t R, int32_t n_top, int32_t *top_rows, float *top_ecpm, hipStream_t s) {
  if (Q <= 0) return hipSuccess;
  hipLaunchKernelGGL(topn_kernel, dim3((unsigned)Q), dim3(kTopnThreads), 0, s, scores, bids, req_off,
                     R, n_top, top_rows, top_ecpm);
  return hipGetLastError();
}

}  // namespace cold

extern "C" int cold_select_topn(const float *scores, const float *bids, const int32_t *req_off,
                                int64_t n_requests, int64_t n_rows, int32_t n_top,
                                int32_t *top_rows, float *top_ecpm, void *stream) {
  if (n_requests < 0 || n_rows < 0 || n_requests > 0x7fffffff || n_rows > 0x7fffffff ||
      n_top < 1 || n_top > COLD_TOPN_MAX)
    return COLD_ERR_INVALID_ARG;
  if (n_requests == 0) return COLD_OK;
  if (!req_off || !top_rows || (n_rows > 0 && (!scores || !bids))) return COLD_ERR_INVALID_ARG;
  const hipError_t e = cold::launch_topn(scores, bids, req_off, n_requests, n_rows, n_top, top_rows,
                                         top_ecpm, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? COLD_OK : COLD_ERR_HIP;
}
