// gather.hip -- embedding gather, sum-pooling, SE weighting, top-k group
// mask and linear_log for the COLD scoring path on gfx950.
//
//  user_pool   one workgroup per request: user-side groups (single-valued
//              and sum-pooled behaviour sequences, Section 3.3) are gathered
//              once per request into fp32 and broadcast to every candidate
//              row of the request later (Section 3.3, parallelism: user
//              features are shared by the ads of a query).
//  gather_se   each wave owns a few consecutive rows and synchronises only
//              within itself.  Ids are read field by field (the column
//              layout of Section 3.3); each lane then owns 16-byte chunks of
//              the wave's network input, laid out so that the wave's output
//              is one contiguous, fully coalesced region.  Chunks hold the
//              gathered embedding in registers while the squeeze (group
//              mean), the two SE layers and the sigmoid (Section 3.2, Eq. 2)
//              run from LDS; the chunks are then reweighted by s_g
//              (Section 3.2), optionally passed through linear_log (Eq. 3)
//              in fp32, and rounded once to the storage type.
//  group_mask  per-request mean importance of each group over the request's
//              rows, then the top-k groups (Section 3.2, feature group
//              selection); ties go to the lower group index.
#include <mutex>
#include <type_traits>
#include <utility>
#include <vector>

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

// Eq. 3: identity on [-1, 1], sign(x) (1 + ln|x|) outside, branch-free.  The
// natural log comes from the hardware log2 (relative error near 2^-22),
// far below the half-precision rounding that follows it.
__device__ __forceinline__ float linear_log(float x) {
  const float ax = fabsf(x);
  const float l = __logf(ax) + 1.0f;   // used only when |x| > 1
  return ax > 1.0f ? copysignf(l, x) : x;
}

__global__ void clear_flag_kernel(int32_t *err) { *err = 0; }

// ------------------------------------------------------------- user_pool
template <typename TS, bool HASHED>
__global__ __launch_bounds__(256) void user_pool_kernel(GatherArgs a) {
  const int64_t q = blockIdx.x;
  const int64_t Q = a.Q;
  const int d = a.d, nu = a.n_user, ns = a.n_seq, nus = nu + ns;
  extern __shared__ float s_u[];   // [nus][d] pooled rows of this request
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
    const TS v = row >= 0 ? tab[(int64_t)row * d + k] : Elem<TS>::from_f32(0.0f);
    a.U[(q * nus + f) * d + k] = Elem<TS>::to_f32(v);
    s_u[f * d + k] = Elem<TS>::to_f32(v);
    static_cast<TS *>(a.Uh)[(q * nu + f) * d + k] = v;   // exact copy in the storage type
    if (k == 0) a.urow[q * nu + f] = row;
  }
  for (int it = threadIdx.x; it < ns * d; it += blockDim.x) {
    const int f = it / d, k = it - f * d, g = nu + f;
    int64_t lo = a.seq_off[f * Q + q], hi = a.seq_off[f * Q + q + 1];
    lo = lo < 0 ? 0 : (lo > a.n_seq_ids ? a.n_seq_ids : lo);
    hi = hi < lo ? lo : (hi > a.n_seq_ids ? a.n_seq_ids : hi);
    const TS *tab = static_cast<const TS *>(a.tables[g]);
    const int64_t rows_g = a.table_rows[g];
    const uint64_t magic_g = a.table_magic[g];
    // sum-pooling in sequence order; ids, rows and values are fetched 16 at
    // a time so that a sequence costs a few memory round trips, not two per id
    constexpr int kSeqBlock = 16;
    float acc = 0.0f;
    bool bad = false;
    for (int64_t j0 = lo; j0 < hi; j0 += kSeqBlock) {
      int32_t row[kSeqBlock];
#pragma unroll
      for (int u = 0; u < kSeqBlock; ++u) {
        const bool in = j0 + u < hi;
        const int64_t j = in ? j0 + u : hi - 1;   // loads stay in range; the result is dropped
        if constexpr (HASHED) {
          const uint64_t raw = static_cast<const uint64_t *>(a.seq_ids)[j];
          const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
          const int32_t r = (int32_t)mod_barrett(mix64(raw ^ salt), (uint64_t)rows_g, magic_g);
          row[u] = in ? r : -1;
        } else {
          const int32_t id = static_cast<const int32_t *>(a.seq_ids)[j];
          const bool ok = id >= 0 && (int64_t)id < rows_g;
          bad |= in && !ok;
          row[u] = in && ok ? id : -1;
        }
      }
      float v[kSeqBlock];   // dropped ids read row 0 (always present) and are not added
#pragma unroll
      for (int u = 0; u < kSeqBlock; ++u)
        v[u] = Elem<TS>::to_f32(tab[(int64_t)(row[u] >= 0 ? row[u] : 0) * d + k]);
#pragma unroll
      for (int u = 0; u < kSeqBlock; ++u)
        if (row[u] >= 0) acc += v[u];
    }
    if (bad) atomicOr(a.err, 1);
    a.U[(q * nus + g) * d + k] = acc;
    s_u[g * d + k] = acc;
  }
  __syncthreads();
  for (int g = threadIdx.x; g < nus; g += blockDim.x) {  // squeeze: mean over d
    float acc = 0.0f;
    for (int k = 0; k < d; ++k) acc += s_u[g * d + k];
    a.zU[q * nus + g] = acc / (float)d;
  }
}

// ------------------------------------------------------------- gather_se
// All synchronisation inside a wave: each wave owns Tw consecutive rows and
// moves on without block barriers, so the 16 waves of a CU overlap their
// gathers freely.  Lane l of a wave owns chunks l, l+64, ... of the wave's
// contiguous output region (Tw rows x M*d elements, 16 bytes per chunk), so
// the final store is coalesced; table chunks are held raw (4 VGPRs) between
// the gather and the reweighting.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

template <typename TS, int MODE, bool LL, bool HASHED, int CPT, bool SE_LDS>
__global__ __launch_bounds__(kGatherThreads, CPT <= 8 ? 4 : 2) void gather_se_kernel(GatherArgs a) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;
  constexpr int EPC = Elem<TS>::kPerChunk;  // elements per 16-byte chunk
  constexpr int IDMAX = kGatherMaxIdsPerLane;
  extern __shared__ __align__(16) unsigned char smem[];

  const int M = a.M, d = a.d, H = a.H;
  const int Mp = a.Mp, Hp = a.Hp;          // padded LDS row strides (z, hidden, SE weights)
  const int nus = a.n_user + a.n_seq, nax = a.n_ad + a.n_cross;
  const int Tw = a.rows_per_tile;          // rows per wave
  const int CPG = d / EPC;                 // chunks per group (power of two)
  const int CPR = M * CPG;                 // chunks per row
  const int lcpg = __builtin_ctz(CPG);
  const float inv_d = 1.0f / (float)d;     // exact: d is a power of two
  const int64_t R = a.R, Q = a.Q;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // (row, chunk) of this lane's first chunk; later chunks step by 64 =
  // q64 rows + r64 chunks, so one step wraps at most once more
  const int t_first = lane / CPR, c_first = lane - t_first * CPR;
  const int q64 = 64 / CPR, r64 = 64 - q64 * CPR;
  auto advance = [&](int &t, int &c) {
    c += r64;
    t += q64;
    const bool wrap = c >= CPR;
    c = wrap ? c - CPR : c;
    t = wrap ? t + 1 : t;
  };

  // ---- block-wide: per-group table metadata and (when small) SE parameters in LDS
  unsigned char *cursor = smem;
  uint64_t *s_tab = reinterpret_cast<uint64_t *>(cursor);   // [M] table base addresses
  uint64_t *s_magic = s_tab + M;                           // [M] Barrett constants
  int32_t *s_rows = reinterpret_cast<int32_t *>(s_magic + M);  // [M] table rows
  int32_t *s_pair = s_rows + M;   // [n_cross] user field | ad field << 16 (GPU cross features)
  cursor += a.meta_lds_bytes;
  for (int g = threadIdx.x; g < M; g += kGatherThreads) {
    s_tab[g] = reinterpret_cast<uint64_t>(a.tables[g]);
    s_magic[g] = a.table_magic[g];
    s_rows[g] = (int32_t)a.table_rows[g];
  }
  const bool gpu_cross = a.cross_pairs != nullptr;
  if (gpu_cross)
    for (int f = threadIdx.x; f < a.n_cross; f += kGatherThreads)
      s_pair[f] = a.cross_pairs[2 * f] | (a.cross_pairs[2 * f + 1] << 16);
  // request offsets in LDS when they fit: the row -> request search then
  // costs LDS latency, not a chain of dependent global loads
  int32_t *s_req = reinterpret_cast<int32_t *>(cursor);   // [Q+1] if req_in_lds
  const bool req_in_lds = a.req_lds_bytes != 0;
  if (req_in_lds)
    for (int64_t i = threadIdx.x; i <= Q; i += kGatherThreads) s_req[i] = a.req_off[i];
  cursor += a.req_lds_bytes;
  // few requests without sequences: their single-valued user rows are
  // resolved and staged in LDS (storage type) here, and no pooling pass runs
  int32_t *s_urow = reinterpret_cast<int32_t *>(cursor);                       // [n_user][Q]
  uint4 *s_uval = reinterpret_cast<uint4 *>(cursor + a.urow_lds_bytes);        // [Q][n_user][CPG]
  const bool users_in_lds = a.users_in_lds != 0;
  if (users_in_lds) {
    const int64_t n_chunks = Q * a.n_user * CPG;
    for (int64_t i = threadIdx.x; i < n_chunks; i += kGatherThreads) {
      const int p = (int)(i & (CPG - 1));
      const int64_t qf = i >> lcpg, q = qf / a.n_user;
      const int f = (int)(qf - q * a.n_user);
      const int32_t row = resolve_row<HASHED>(a.user_ids, (int64_t)f * Q + q, f, a.table_rows[f],
                                              a.table_magic[f], a.err);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0) v = reinterpret_cast<const uint4 *>(static_cast<const TS *>(a.tables[f]) + (int64_t)row * d)[p];
      s_uval[i] = v;
      if (p == 0) s_urow[(int64_t)f * Q + q] = row;
    }
    if constexpr (MODE != kApplyWeights) {   // request offsets sanity, otherwise done by the pooling pass
      for (int64_t q = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x; q < Q;
           q += (int64_t)gridDim.x * kGatherThreads) {
        bool bad = a.req_off[q + 1] < a.req_off[q];
        if (q == 0) bad |= a.req_off[0] != 0;
        if (q == Q - 1) bad |= (int64_t)a.req_off[Q] != R;
        if (bad) atomicOr(a.err, 2);
      }
    }
  }
  cursor += a.urow_lds_bytes + a.uval_lds_bytes;
  const float *w1 = a.w1, *b1 = a.b1, *w2 = a.w2, *b2 = a.b2;
  if constexpr ((MODE == kFull || MODE == kWeightsOnly) && SE_LDS) {
    {
      // W1 [H][Mp], W2 [M][Hp] (rows 16-byte aligned, padding zero), b1 [H], b2 [M]
      float *sw = reinterpret_cast<float *>(cursor);
      float *sw2 = sw + H * Mp, *sb1 = sw2 + M * Hp, *sb2 = sb1 + H;
      for (int i = threadIdx.x; i < H * Mp; i += kGatherThreads) {
        const int j = i / Mp, g = i - j * Mp;
        sw[i] = g < M ? a.w1[j * M + g] : 0.0f;
      }
      for (int i = threadIdx.x; i < M * Hp; i += kGatherThreads) {
        const int g = i / Hp, j = i - g * Hp;
        sw2[i] = j < H ? a.w2[g * H + j] : 0.0f;
      }
      for (int i = threadIdx.x; i < H; i += kGatherThreads) sb1[i] = a.b1[i];
      for (int i = threadIdx.x; i < M; i += kGatherThreads) sb2[i] = a.b2[i];
      w1 = sw; b1 = sb1; w2 = sw2; b2 = sb2;
      cursor += a.se_lds_bytes;
    }
  }
  __syncthreads();  // the only block-wide barrier

  unsigned char *wb = cursor + (size_t)wave * a.wave_lds_bytes;
  const int ns = a.n_seq, nu = a.n_user;
  // 16-byte aligned first: z and hid are read as float4 rows
  float *z = reinterpret_cast<float *>(wb);                // [Tw][Mp] squeeze
  float *hid = z + Tw * Mp;                                // [Tw][Hp] SE hidden layer
  float *ust = hid + Tw * Hp;                              // [Tw][ns*d] pooled sequence rows
  float *sv = ust + Tw * ns * d;                           // [Tw][M] SE weights
  int32_t *ridx = reinterpret_cast<int32_t *>(sv + Tw * M);  // [Tw][nax]
  int32_t *rq = ridx + Tw * nax;                           // [Tw]
  const TS *Uh = static_cast<const TS *>(a.Uh);

  // persistent: each wave walks the row tiles wave_id, wave_id + waves, ...
  const int64_t n_tiles = (R + Tw - 1) / Tw;
  const int64_t stride = (int64_t)gridDim.x * (kGatherThreads / 64);
  for (int64_t wt = (int64_t)blockIdx.x * (kGatherThreads / 64) + wave; wt < n_tiles; wt += stride) {
  const int64_t r0 = wt * Tw;
  // rows of this tile that exist: t < tv is t < Tw && r0 + t < R
  const int tv = R - r0 < Tw ? (int)(R - r0) : Tw;
  // chunk coordinates, opaque to the compiler so that nothing derived from
  // them is hoisted out of the tile loop (which would pin registers)
  int tf = t_first, cf = c_first, ln = lane;
  asm volatile("" : "+v"(tf), "+v"(cf), "+v"(ln));

  // ---- ad/cross ids first (all loads issued before any is used; they go
  //      to registers, so they need not wait for the previous tile), then
  //      the request of each row, then table rows
  typedef typename std::conditional<HASHED, uint64_t, int32_t>::type id_t;
  id_t idv[IDMAX];
#pragma unroll
  for (int k = 0; k < IDMAX; ++k) {
    const int i = ln + 64 * k;
    idv[k] = 0;
    if (i < Tw * nax) {
      const int f = fast_div(i, a.mg_tw), t = i - f * Tw;
      const int64_t r = r0 + t;
      if (r < R) {
        const bool is_ad = f < a.n_ad;
        // a cross field built on the GPU starts from its ad field's id
        const int fa = is_ad ? f : (gpu_cross ? s_pair[f - a.n_ad] >> 16 : f - a.n_ad);
        const id_t *ids = static_cast<const id_t *>(is_ad || gpu_cross ? a.ad_ids : a.cross_ids);
        idv[k] = ids[(int64_t)fa * R + r];
      }
    }
  }
  wave_sync();  // the previous tile's LDS reads are done
  for (int t = ln; t < Tw; t += 64) {
    const int64_t r = r0 + t;
    int32_t q = 0;
    if (r < R) q = (int32_t)(req_in_lds ? request_of_row(s_req, Q, r) : request_of_row(a.req_off, Q, r));
    rq[t] = q;
  }
  wave_sync();  // rq visible
#pragma unroll
  for (int k = 0; k < IDMAX; ++k) {
    const int i = ln + 64 * k;
    if (i < Tw * nax) {
      const int f = fast_div(i, a.mg_tw), t = i - f * Tw;
      const int64_t r = r0 + t;
      const int g = nus + f;
      int32_t row = -1;
      if (r < R) {
        bool keep = true;
        if constexpr (MODE == kApplyWeights) keep = !a.mask || a.mask[(int64_t)rq[t] * M + g] != 0;
        if (gpu_cross && f >= a.n_ad) {
          // user x ad cross value: key = mix64(user id) ^ ad id, hashed into
          // the group's table (ids as their unsigned bit patterns)
          const int fu = s_pair[f - a.n_ad] & 0xFFFF;
          const id_t *uids = static_cast<const id_t *>(a.user_ids);
          uint64_t uid, aid;
          if constexpr (HASHED) {
            uid = (uint64_t)uids[(int64_t)fu * Q + rq[t]];
            aid = (uint64_t)idv[k];
          } else {
            uid = (uint64_t)(uint32_t)uids[(int64_t)fu * Q + rq[t]];
            aid = (uint64_t)(uint32_t)idv[k];
          }
          const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
          row = (int32_t)mod_barrett(mix64((mix64(uid) ^ aid) ^ salt), (uint64_t)s_rows[g], s_magic[g]);
        } else if constexpr (HASHED) {
          const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
          row = (int32_t)mod_barrett(mix64((uint64_t)idv[k] ^ salt), (uint64_t)s_rows[g], s_magic[g]);
        } else {
          row = (int32_t)idv[k];
          if (row < 0 || row >= s_rows[g]) {
            atomicOr(a.err, 1);
            row = -1;
          }
        }
        if (!keep) row = -1;
        if (MODE != kApplyWeights && a.rows_out) a.rows_out[(int64_t)g * R + r] = row;
      }
      ridx[t * nax + f] = row;
    }
  }
  // ---- pooled sequence rows of the wave's rows into LDS (fp32: sums can
  //      exceed the storage range), squeeze of the user groups
  const int sd4 = ns * d / 4;
  for (int i = ln; i < Tw * sd4; i += 64) {
    const int t = fast_div(i, a.mg_sd4), k4 = i - t * sd4;
    reinterpret_cast<float4 *>(ust)[i] =
        reinterpret_cast<const float4 *>(a.U + ((int64_t)rq[t] * nus + nu) * d)[k4];
  }
  if constexpr (MODE == kFull || MODE == kWeightsOnly || MODE == kSqueezeRaw) {   // squeeze of the pooled sequences
    for (int i = ln; i < Tw * ns; i += 64) {
      const int t = fast_div(i, a.mg_ns), g = nu + (i - t * ns);
      z[t * Mp + g] = r0 + t < R ? a.zU[(int64_t)rq[t] * nus + g] : 0.0f;
    }
  }
  wave_sync();
  if (MODE != kApplyWeights && a.rows_out) {
    for (int i = ln; i < Tw * nus; i += 64) {
      const int f = fast_div(i, a.mg_tw), t = i - f * Tw;
      const int64_t r = r0 + t;
      if (r < R)
        a.rows_out[(int64_t)f * R + r] =
            f >= nu ? -1 : users_in_lds ? s_urow[(int64_t)f * Q + rq[t]] : a.urow[(int64_t)rq[t] * nu + f];
    }
  }

  // ---- gather every chunk first (all loads in flight): table rows, and the
  //      request's single-valued user rows (storage type), then squeeze
  uint4 raw[CPT];
  {
    int t = tf, c = cf;
    asm volatile("" : "+v"(t), "+v"(c));   // recomputed per phase, not kept live
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      const int g = c >> lcpg, p = c & (CPG - 1);
      raw[j] = make_uint4(0, 0, 0, 0);
      if (t < tv && (g < nu || g >= nus)) {
        uint64_t addr = 0;
        if (g < nu) {
          bool keep = true;
          if constexpr (MODE == kApplyWeights) keep = !a.mask || a.mask[(int64_t)rq[t] * M + g] != 0;
          if (keep && users_in_lds) raw[j] = s_uval[((int64_t)rq[t] * nu + g) * CPG + p];
          else if (keep) addr = reinterpret_cast<uint64_t>(Uh + ((int64_t)rq[t] * nu + g) * d + p * EPC);
        } else {
          const int32_t row = ridx[t * nax + (g - nus)];
          if (row >= 0) addr = s_tab[g] + ((uint64_t)row * d + p * EPC) * sizeof(TS);
        }
        if (addr) {
          const u32x4 w = *reinterpret_cast<gl_u32x4 *>(addr);
          raw[j] = make_uint4(w.x, w.y, w.z, w.w);
        }
      }
      advance(t, c);
    }
  }
  if constexpr (MODE == kFull || MODE == kWeightsOnly || MODE == kSqueezeRaw) {
    int t = tf, c = cf;
    asm volatile("" : "+v"(t), "+v"(c));   // recomputed per phase, not kept live
#pragma unroll
    for (int j = 0; j < CPT; ++j, advance(t, c)) {
      const int g = c >> lcpg, p = c & (CPG - 1);
      float v[EPC];
      Elem<TS>::unpack(raw[j], v);
      float part = 0.0f;
#pragma unroll
      for (int e = 0; e < EPC; ++e) part += v[e];
      // butterfly over the CPG lanes of the group (offsets are constants;
      // CPG <= 64 is a power of two)
      if (CPG > 1) part += __shfl_xor(part, 1);
      if (CPG > 2) part += __shfl_xor(part, 2);
      if (CPG > 4) part += __shfl_xor(part, 4);
      if (CPG > 8) part += __shfl_xor(part, 8);
      if (CPG > 16) part += __shfl_xor(part, 16);
      if (CPG > 32) part += __shfl_xor(part, 32);
      if (t < Tw && p == 0 && (g < nu || g >= nus)) z[t * Mp + g] = t < tv ? part * inv_d : 0.0f;
    }
    wave_sync();

    if constexpr (MODE == kSqueezeRaw) {
      // the squeeze [R][M] and the gathered rows, exact in the storage type,
      // into the network input's place, for the separate SE and apply passes
      for (int it = ln; it < Tw * M; it += 64) {
        const int t = fast_div(it, a.mg_m), g = it - t * M;
        if (r0 + t < R) a.z_out[r0 * M + it] = z[t * Mp + g];
      }
      TS *X = static_cast<TS *>(a.X);
      int t = tf, c = cf;
      asm volatile("" : "+v"(t), "+v"(c));
#pragma unroll
      for (int j = 0; j < CPT; ++j, advance(t, c)) {
        const int i = ln + 64 * j;
        if (t < tv) *reinterpret_cast<uint4 *>(X + (r0 * CPR + i) * EPC) = raw[j];
      }
    } else {
    // ---- SE block of the wave's rows (Eq. 2)
    // sums from the bias in index order; from LDS, weight and input rows are
    // read four at a time (rows padded to Mp / Hp); from global memory, the
    // weights are read transposed, so that the lanes (one output each) of a
    // step read consecutive words
    for (int it = ln; it < Tw * H; it += 64) {
      const int t = fast_div(it, a.mg_h), jh = it - t * H;
      const float *zt = z + t * Mp;
      float acc = b1[jh];
      if constexpr (SE_LDS) {
        const float *w = w1 + jh * Mp;
        int g = 0;
#pragma unroll 1
        for (; g + 4 <= M; g += 4) {
          const float4 wv = *reinterpret_cast<const float4 *>(w + g);
          const float4 zv = *reinterpret_cast<const float4 *>(zt + g);
          acc += wv.x * zv.x;
          acc += wv.y * zv.y;
          acc += wv.z * zv.z;
          acc += wv.w * zv.w;
        }
        for (; g < M; ++g) acc += w[g] * zt[g];
      } else {
        // W1 transposed ([M][H]): the lanes of a step read consecutive words
        const float *w = a.w1t + jh;
#pragma unroll 8
        for (int g = 0; g < M; ++g) acc += w[g * H] * zt[g];
      }
      hid[t * Hp + jh] = acc > 0.0f ? acc : 0.0f;
    }
    wave_sync();
    for (int it = ln; it < Tw * M; it += 64) {
      const int t = fast_div(it, a.mg_m), g = it - t * M;
      const float *ht = hid + t * Hp;
      float acc = b2[g];
      if constexpr (SE_LDS) {
        const float *w = w2 + g * Hp;
        int jh = 0;
#pragma unroll 1
        for (; jh + 4 <= H; jh += 4) {
          const float4 wv = *reinterpret_cast<const float4 *>(w + jh);
          const float4 hv = *reinterpret_cast<const float4 *>(ht + jh);
          acc += wv.x * hv.x;
          acc += wv.y * hv.y;
          acc += wv.z * hv.z;
          acc += wv.w * hv.w;
        }
        for (; jh < H; ++jh) acc += w[jh] * ht[jh];
      } else {
        // W2 transposed ([H][M]): the lanes of a step read consecutive words
        const float *w = a.w2t + g;
#pragma unroll 8
        for (int jh = 0; jh < H; ++jh) acc += w[jh * M] * ht[jh];
      }
      const float sg = 1.0f / (1.0f + expf(-acc));
      sv[it] = sg;
      if (a.s_buf && r0 + t < R) a.s_buf[r0 * M + it] = sg;
    }
    }   // SE block
  } else if constexpr (MODE == kApplyWeights) {
    for (int it = ln; it < Tw * M; it += 64) {
      const int t = fast_div(it, a.mg_m), g = it - t * M;
      float sg = 0.0f;
      if (r0 + t < R && (!a.mask || a.mask[(int64_t)rq[t] * M + g])) sg = a.s_buf[r0 * M + it];
      sv[it] = sg;
    }
  }
  if constexpr (MODE == kRawOut) {
  // ---- the concatenated embedding itself, in fp32 (pooled sequence groups
  //      are fp32 sums), for an SE computed by a separate dense layer
  float *E = static_cast<float *>(a.X);
  int t = tf, c = cf;
  asm volatile("" : "+v"(t), "+v"(c));   // recomputed per phase, not kept live
#pragma unroll
  for (int j = 0; j < CPT; ++j, advance(t, c)) {
    const int i = ln + 64 * j;
    const int g = c >> lcpg, p = c & (CPG - 1);
    if (t < tv) {
      float v[EPC];
      if (g >= nu && g < nus) {
        const float *src = ust + t * ns * d + (g - nu) * d + p * EPC;
#pragma unroll
        for (int e = 0; e < EPC; ++e) v[e] = src[e];
      } else {
        Elem<TS>::unpack(raw[j], v);
      }
      float4 *dst = reinterpret_cast<float4 *>(E + (r0 * CPR + i) * EPC);
#pragma unroll
      for (int e = 0; e < EPC / 4; ++e) dst[e] = make_float4(v[4 * e], v[4 * e + 1], v[4 * e + 2], v[4 * e + 3]);
    }
  }
  }
  if constexpr (MODE == kFull || MODE == kApplyWeights) {
  wave_sync();

  // ---- reweight, linear_log, round once, coalesced store
  TS *X = static_cast<TS *>(a.X);
  int t = tf, c = cf;
  asm volatile("" : "+v"(t), "+v"(c));   // recomputed per phase, not kept live
#pragma unroll
  for (int j = 0; j < CPT; ++j, advance(t, c)) {
    const int i = ln + 64 * j;
    const int g = c >> lcpg, p = c & (CPG - 1);
    if (t < tv) {
      const float sg = sv[t * M + g];
      float v[EPC];
      if (g >= nu && g < nus) {
        const float *src = ust + t * ns * d + (g - nu) * d + p * EPC;
#pragma unroll
        for (int e = 0; e < EPC; ++e) v[e] = src[e];
      } else {
        Elem<TS>::unpack(raw[j], v);
      }
      float o[EPC];
#pragma unroll
      for (int e = 0; e < EPC; ++e) {
        const float x = sg * v[e];
        o[e] = LL ? linear_log(x) : x;
      }
      *reinterpret_cast<uint4 *>(X + (r0 * CPR + i) * EPC) = Elem<TS>::pack(o);
    }
  }
  }
  }  // tile loop
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
#pragma unroll 8
    for (int64_t r = a; r < b; ++r) acc += s_buf[r * M + g];
    partial[(q * P + p) * M + g] = acc;
  }
}

// Per request: importance I_g = (sum of the P partial sums of group g) / n,
// then the top-k mask. The partial sums are added by kSelQuarters threads per
// group, each over a contiguous quarter of the parts, and the quarters are
// added in order, so the result does not depend on the launch.
constexpr int kSelQuarters = 4;
__global__ __launch_bounds__(1024) void mask_select_kernel(const float *partial, const int32_t *req_off,
                                                           int64_t R, int32_t M, int32_t P, int32_t k,
                                                           uint8_t *mask, uint8_t *mask_out) {
  extern __shared__ float lds[];  // [kSelQuarters][M] quarter sums, then [M] importance
  float *imp = lds + kSelQuarters * M;
  const int64_t q = blockIdx.x;
  int64_t lo = req_off[q], hi = req_off[q + 1];
  lo = lo < 0 ? 0 : (lo > R ? R : lo);
  hi = hi < lo ? lo : (hi > R ? R : hi);
  const float n = (float)(hi - lo);
  const int per = P / kSelQuarters;
  for (int idx = threadIdx.x; idx < kSelQuarters * M; idx += blockDim.x) {
    const int c = idx / M, g = idx - c * M;
    const float *src = partial + (q * P + c * per) * M + g;
    float acc = 0.0f;
#pragma unroll 16
    for (int p = 0; p < per; ++p) acc += src[(int64_t)p * M];
    lds[idx] = acc;
  }
  __syncthreads();
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    float acc = lds[g];
#pragma unroll
    for (int c = 1; c < kSelQuarters; ++c) acc += lds[c * M + g];
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

// The same importance and mask from the row-wise SE's 16-row tile sums:
// request q adds, per group, the rows before its first whole tile, the sums
// of its whole tiles in P contiguous parts (P threads per group or per four
// groups, whose loads are all in flight together; the parts added in order)
// and the rows after its last whole tile, in that order, so the result does
// not depend on the launch.
// parts of the tile sums: the block's threads but the last M (which add the
// rows outside whole tiles) over the groups, one or four groups per thread
__host__ __device__ inline int mask_tile_parts(int M) {
  const int nq = M % 4 == 0 ? M / 4 : M;   // threads per part
  const int p = (1024 - M) / nq;
  return p < 1 ? 1 : (p > 64 ? 64 : p);
}

__global__ __launch_bounds__(1024) void mask_select_tiles_kernel(const float *s_buf,
                                                                 const float *tpart,
                                                                 const int32_t *req_off, int64_t R,
                                                                 int32_t M, int32_t k, uint8_t *mask,
                                                                 uint8_t *mask_out, int32_t *kept) {
  extern __shared__ float lds[];  // [P][M] part sums, [M] importance, [M] ranks, [2][M] edges
  __shared__ int32_t s_wkept[4];  // kept groups per wave of the first 256 threads
  const int P = mask_tile_parts(M);
  float *imp = lds + P * M;
  int *rank = reinterpret_cast<int *>(imp + M);
  const int64_t q = blockIdx.x;
  int64_t lo = req_off[q], hi = req_off[q + 1];
  lo = lo < 0 ? 0 : (lo > R ? R : lo);
  hi = hi < lo ? lo : (hi > R ? R : hi);
  const float n = (float)(hi - lo);
  const int64_t t0 = (lo + 15) / 16, t1 = hi / 16;   // whole tiles [t0, t1)
  const bool whole = t0 < t1;
  // rows outside whole tiles: fewer than 32 before them (all rows when there
  // are none), fewer than 16 after them
  const int64_t head_end = whole ? 16 * t0 : hi, tail_begin = whole ? 16 * t1 : hi;
  const int64_t nt = whole ? t1 - t0 : 0, per = (nt + P - 1) / P;
  const bool v4 = M % 4 == 0;
  const int nq = v4 ? M / 4 : M;
  for (int idx = threadIdx.x; idx < P * nq; idx += (int)blockDim.x - M) {
    const int p = idx / nq, gq = idx - p * nq;
    const int64_t a = t0 + p * per, b = a + per < t0 + nt ? a + per : t0 + nt;
    // blocks of 16 tiles: every load of a block in flight before its sums,
    // which run in tile order (the block's slots past b add +0 to a sum of
    // non-negative weights, which leaves it unchanged)
    if (v4) {
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int64_t t = a; t < b; t += 16) {
        float4 v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          v[i] = t + i < b ? reinterpret_cast<const float4 *>(tpart + (t + i) * M)[gq]
                           : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          acc.x += v[i].x; acc.y += v[i].y; acc.z += v[i].z; acc.w += v[i].w;
        }
      }
      reinterpret_cast<float4 *>(lds + p * M)[gq] = acc;
    } else {
      float acc = 0.0f;
      for (int64_t t = a; t < b; t += 16) {
        float v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = t + i < b ? tpart[(t + i) * M + gq] : 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) acc += v[i];
      }
      lds[p * M + gq] = acc;
    }
  }
  // the rows outside whole tiles, summed in row order by the last M threads
  // of the block while the others add the tiles (every load in flight first)
  float *edge = reinterpret_cast<float *>(rank + M);   // [2][M] head and tail sums
  for (int g = (int)threadIdx.x - ((int)blockDim.x - M); g >= 0; g = -1) {
    float hv[32], tv[16];
#pragma unroll
    for (int i = 0; i < 32; ++i) hv[i] = lo + i < head_end ? s_buf[(lo + i) * M + g] : 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) tv[i] = tail_begin + i < hi ? s_buf[(tail_begin + i) * M + g] : 0.0f;
    float h = 0.0f, t = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) h += hv[i];
#pragma unroll
    for (int i = 0; i < 16; ++i) t += tv[i];
    edge[g] = h;
    edge[M + g] = t;
  }
  for (int g = threadIdx.x; g < M; g += blockDim.x) rank[g] = 0;
  __syncthreads();
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    float acc = edge[g];
    for (int p = 0; p < P; ++p) acc += lds[p * M + g];
    acc += edge[M + g];
    imp[g] = n > 0.0f ? acc / n : 0.0f;
  }
  __syncthreads();
  // rank of group g: groups ahead of it, counted by several threads over
  // blocks of the others (integer sums: any order gives the same count)
  const int RP = (int)(blockDim.x / M) < 1 ? 1 : (int)(blockDim.x / M);
  const int rper = (M + RP - 1) / RP;
  for (int idx = threadIdx.x; idx < RP * M; idx += blockDim.x) {
    const int rp = idx / M, g = idx - rp * M;
    const float ig = imp[g];
    const int o0 = rp * rper, o1 = o0 + rper < M ? o0 + rper : M;
    int cnt = 0;
    for (int o = o0; o < o1; ++o) {
      const float io = imp[o];
      cnt += (io > ig || (io == ig && o < g)) ? 1 : 0;
    }
    atomicAdd(&rank[g], cnt);
  }
  __syncthreads();
  for (int g = threadIdx.x; g < M; g += blockDim.x) {
    const uint8_t keep = rank[g] < k ? 1 : 0;
    mask[q * M + g] = keep;
    if (mask_out) mask_out[q * M + g] = keep;
  }
  if (kept) {
    // the kept groups in group order, min(k, M) of them: thread g < 256
    // takes group g (M <= 256), its place is the count of kept groups
    // before it (wave ballots, then the earlier waves' counts)
    const int g = threadIdx.x, lane = g & 63, w = g >> 6;
    const bool f = g < M && rank[g] < k;
    unsigned long long bal = 0;
    if (g < 256) {
      bal = __ballot(f);
      if (lane == 0) s_wkept[w] = __popcll(bal);
    }
    __syncthreads();
    const int kp = k < M ? k : M;
    if (f) {
      int pos = __popcll(bal & ((1ull << lane) - 1));
      for (int v = 0; v < w; ++v) pos += s_wkept[v];
      if (pos < kp) kept[q * kp + pos] = g;
    }
    // ranks form a permutation unless an importance is NaN; then the list
    // is still filled with valid groups
    const int n_kept = s_wkept[0] + s_wkept[1] + s_wkept[2] + s_wkept[3];
    for (int j = n_kept + (int)threadIdx.x; j < kp; j += (int)blockDim.x) kept[q * kp + j] = 0;
  }
}

hipError_t launch_group_mask_tiles(const float *s_buf, const float *tile_part,
                                   const int32_t *req_off, int64_t Q, int64_t R, int32_t M,
                                   int32_t k, uint8_t *mask, uint8_t *mask_out, int32_t *kept,
                                   hipStream_t s) {
  if (Q <= 0) return hipSuccess;
  if (M % 4 == 0 && (reinterpret_cast<uintptr_t>(tile_part) & 15)) return hipErrorInvalidValue;
  if (kept && (M > 256 || k <= 0)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mask_select_tiles_kernel, dim3((unsigned)Q), dim3(1024),
                     sizeof(float) * (size_t)(mask_tile_parts(M) + 4) * M, s, s_buf, tile_part,
                     req_off, R, M, k, mask, mask_out, kept);
  return hipGetLastError();
}

// ------------------------------------------------------------- launchers
template <typename TS>
static hipError_t user_pool_t(bool hashed, const GatherArgs &a, hipStream_t s) {
  // a row holds at most kGatherMaxChunksPerRow chunks, so nus * d floats fit in LDS
  const size_t shmem = sizeof(float) * (size_t)(a.n_user + a.n_seq) * a.d;
  if (hashed) hipLaunchKernelGGL((user_pool_kernel<TS, true>), dim3(a.Q), dim3(256), shmem, s, a);
  else hipLaunchKernelGGL((user_pool_kernel<TS, false>), dim3(a.Q), dim3(256), shmem, s, a);
  return hipGetLastError();
}

bool user_pool_needed(int dtype, const GatherArgs &a) {
  if (a.n_seq > 0) return true;
  const int64_t es = dtype == kF32 ? 4 : 2;
  return (int64_t)a.n_user * a.Q * a.d * es > kGatherMaxUserValLds;
}

hipError_t launch_user_pool(int dtype, bool hashed, const GatherArgs &a, hipStream_t s) {
  if (a.Q <= 0 || !user_pool_needed(dtype, a)) return hipSuccess;
  switch (dtype) {
    case kF32: return user_pool_t<float>(hashed, a, s);
    case kBF16: return user_pool_t<__bf16>(hashed, a, s);
    default: return user_pool_t<_Float16>(hashed, a, s);
  }
}

// CUs of the current device (cached per device)
int device_cus() {
  static std::mutex mu;
  static std::vector<std::pair<int, int>> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lk(mu);
  for (const auto &e : cache)
    if (e.first == dev) return e.second;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  cache.emplace_back(dev, cus);
  return cus;
}

// Resident workgroups of a kernel on the current device (cached): the
// persistent gather launches no more than fit at once.
static int resident_blocks(const void *kernel, size_t shmem) {
  struct Entry { const void *k; size_t sh; int dev; int blocks; };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lk(mu);
  for (const Entry &e : cache)
    if (e.k == kernel && e.sh == shmem && e.dev == dev) return e.blocks;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kGatherThreads, shmem) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const int blocks = per_cu * cus;
  cache.push_back({kernel, shmem, dev, blocks});
  return blocks;
}

// ------------------------------------------------------------- gather_full
// Gather, squeeze, SE and reweighting of a row tile in registers (Section
// 3.2: Eq. 2 read as squeeze -> FC -> ReLU -> FC -> sigmoid, Eq. 3 when LL),
// for models with at most 64 groups, at most 16 hidden SE units, 32-byte
// group rows and no sequence groups.  A tile is 16 rows; lane l = 16 q + c
// of a wave owns row c and groups g = 4 k + q of its slots k: it loads their
// ids and both 16-byte chunks of each group row itself, so a group's squeeze
// is a sum inside one lane, and the lanes' squeeze values are already the B
// operand of a 16x16x4 fp32 MFMA whose K index is g = 4 k + q at step k.
// Layer 1 is one 16-unit hidden block (h^T = W1 z^T); its output fragment
// (units 4 q + e of row c in lane (c, q)) is layer 2's B operand as it
// stands.  Layer 2 forms its output rows in the order g = 16 gb + 4 e + q
// (row 4 q + e of block gb), so the weight of slot k = 4 gb + e lands in the
// lane that holds the group's values.  Both SE matrices are packed in that
// operand order at load time and staged in LDS.  The users' rows come from
// the pooling pass (storage type, one per request), or, for few requests,
// are resolved into LDS by every workgroup.
//   Up to 48 groups, one wave takes a whole tile (12 slots per lane, held in
// registers from the gather to the store).  Above that, a workgroup takes a
// tile with one wave per 16 groups (4 slots per lane); each wave forms
// layer 1's sum over its own slots (wave 0's from b1), the parts are added
// in wave order through LDS, and wave w forms layer 2's block gb = w.
//   Products and sums are fp32; the squeeze and the SE sums run in another
// order than the general gather's index order, which only moves fp32
// rounding.  A row's result does not depend on the other rows of its tile,
// and every batch size of a model takes the same form, so a score does not
// depend on the batch it comes in.
constexpr int kFullMaxM = 64;
constexpr int kFullMaxH = 16;
constexpr int kFullTileM = 48;   // the one-wave-per-tile form up to this many groups

bool gather_full_shape(int32_t M, int32_t H, int32_t row_bytes, int32_t n_seq) {
  return n_seq == 0 && M > 0 && M <= kFullMaxM && H > 0 && H <= kFullMaxH && row_bytes == 32;
}

// every batch size of a supported model takes this kernel, so that a row's
// score does not depend on the batch it comes in
bool gather_full_supported(int dtype, const GatherArgs &a) {
  const int es = dtype == kF32 ? 4 : 2;
  return gather_full_shape(a.M, a.H, a.d * es, a.n_seq) && a.w1f != nullptr && a.w2f != nullptr;
}

// W1f [4][64 lanes][4]: element e of vector (u, lane) is W1[c][4 (4 u + e) + q];
// W2f [4][64 lanes][4]: element e of vector (gb, lane) is
// W2[16 gb + 4 (c & 3) + (c >> 2)][4 q + e]; zero outside M x H
__global__ __launch_bounds__(256) void pack_se_full_kernel(const float *__restrict__ w1,
                                                           const float *__restrict__ w2, int M, int H,
                                                           float *__restrict__ w1f,
                                                           float *__restrict__ w2f) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= 2 * kSeFullFloats) return;
  const int i2 = i % kSeFullFloats;
  const int e = i2 & 3, lane = (i2 >> 2) & 63, blk = i2 >> 8, c = lane & 15, q = lane >> 4;
  if (i < kSeFullFloats) {
    const int g = 4 * (4 * blk + e) + q, j = c;
    w1f[i2] = j < H && g < M ? w1[j * M + g] : 0.0f;
  } else {
    const int g = 16 * blk + 4 * (c & 3) + (c >> 2), j = 4 * q + e;
    w2f[i2] = g < M && j < H ? w2[g * H + j] : 0.0f;
  }
}

hipError_t launch_pack_se_full(const float *w1, const float *w2, int32_t M, int32_t H, float *w1f,
                               float *w2f, hipStream_t s) {
  if (!gather_full_shape(M, H, 32, 0)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_se_full_kernel, dim3((2 * kSeFullFloats + 255) / 256), dim3(256), 0, s, w1,
                     w2, M, H, w1f, w2f);
  return hipGetLastError();
}

// Models of up to 48 groups: one wave per 16-row tile and all its groups,
// NS slots per lane (M <= 4 NS); at 12 slots the group rows of two
// workgroups per CU fit in registers.
template <typename TS, bool LL, bool HASHED, int NS, bool ULDS>
__global__ __launch_bounds__(256, 2) void gather_full_kernel(GatherArgs a) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;
  typedef typename std::conditional<HASHED, uint64_t, int32_t>::type id_t;
  constexpr int EPC = Elem<TS>::kPerChunk;   // elements per 16-byte chunk
  constexpr int EPG = 2 * EPC;               // elements per group (d)
  __shared__ uint64_t s_tab[kFullMaxM];
  __shared__ uint64_t s_magic[kFullMaxM];
  __shared__ int32_t s_rows[kFullMaxM];
  __shared__ int32_t s_pair[kFullMaxM];
  __shared__ int32_t s_req[kGatherMaxReqLds + 1];
  __shared__ float4 s_w1[kSeFullFloats / 4], s_w2[kSeFullFloats / 4];   // packed SE operands
  __shared__ float4 s_b1[4], s_b2[16];   // b1[4 q + e]; b2[16 gb + 4 e + q] at [4 gb + q].e
  extern __shared__ __align__(16) unsigned char s_users[];   // [Q][nu][2] chunks, then [nu][Q] rows
  const int M = a.M, H = a.H, nu = a.n_user, n_ad = a.n_ad;
  const int64_t R = a.R, Q = a.Q;
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int wave = tid >> 6, nt = 256, nw = 4;
  for (int g = tid; g < M; g += nt) {
    s_tab[g] = reinterpret_cast<uint64_t>(a.tables[g]);
    s_magic[g] = a.table_magic[g];
    s_rows[g] = (int32_t)a.table_rows[g];
  }
  const bool gpu_cross = a.cross_pairs != nullptr;
  if (gpu_cross)
    for (int f = tid; f < a.n_cross; f += nt) s_pair[f] = a.cross_pairs[2 * f] | (a.cross_pairs[2 * f + 1] << 16);
  const bool req_in_lds = Q <= kGatherMaxReqLds;
  if (req_in_lds)
    for (int64_t i = tid; i <= Q; i += nt) s_req[i] = a.req_off[i];
  for (int i = tid; i < kSeFullFloats / 4; i += nt) {
    s_w1[i] = reinterpret_cast<const float4 *>(a.w1f)[i];
    s_w2[i] = reinterpret_cast<const float4 *>(a.w2f)[i];
  }
  if (tid < 16) {
    const int j = tid;
    reinterpret_cast<float *>(s_b1)[j] = j < H ? a.b1[j] : 0.0f;
  }
  if (tid < 64) {
    const int gb = tid >> 4, qq = (tid >> 2) & 3, e = tid & 3, g = 16 * gb + 4 * e + qq;
    reinterpret_cast<float *>(s_b2)[tid] = g < M ? a.b2[g] : 0.0f;
  }
  // few requests: their users' rows resolved and staged here (no pooling pass)
  constexpr bool users_lds = ULDS;
  uint4 *s_uval = reinterpret_cast<uint4 *>(s_users);
  int32_t *s_urow = reinterpret_cast<int32_t *>(s_users + (size_t)Q * nu * 32);
  if (users_lds) {
    for (int64_t i = tid; i < Q * nu * 2; i += nt) {
      const int p = (int)(i & 1);
      const int64_t qq = (i >> 1) / nu;
      const int f = (int)((i >> 1) - qq * nu);
      const int32_t row = resolve_row<HASHED>(a.user_ids, (int64_t)f * Q + qq, f, a.table_rows[f],
                                              a.table_magic[f], a.err);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0) v = reinterpret_cast<const uint4 *>(static_cast<const TS *>(a.tables[f]) + (int64_t)row * EPG)[p];
      s_uval[i] = v;
      if (p == 0) s_urow[(int64_t)f * Q + qq] = row;
    }
    // request offsets sanity (the pooling pass checks them otherwise)
    for (int64_t qq = (int64_t)blockIdx.x * nt + tid; qq < Q; qq += (int64_t)gridDim.x * nt) {
      bool bad = a.req_off[qq + 1] < a.req_off[qq];
      if (qq == 0) bad |= a.req_off[0] != 0;
      if (qq == Q - 1) bad |= (int64_t)a.req_off[Q] != R;
      if (bad) atomicOr(a.err, 2);
    }
  }
  __syncthreads();

  const int KS = (M + 3) >> 2, GB = (M + 15) >> 4;   // slots and output blocks in use
  const float inv_d = 1.0f / (float)EPG;             // exact: EPG is a power of two
  const TS *Uh = static_cast<const TS *>(a.Uh);
  TS *X = static_cast<TS *>(a.X);
  const uint64_t dummy = s_tab[0];                   // row 0 of a table: always present

  const int64_t n_tiles = (R + 15) >> 4;
  for (int64_t wt = (int64_t)blockIdx.x * nw + wave; wt < n_tiles; wt += (int64_t)gridDim.x * nw) {
    const int64_t r = wt * 16 + c;
    const bool row_ok = r < R;
    const int64_t rr = row_ok ? r : R - 1;           // clamped: loaded, never stored
    int64_t rq = 0;
    if (nu > 0 || gpu_cross)
      rq = req_in_lds ? request_of_row(s_req, Q, rr) : request_of_row(a.req_off, Q, rr);

    // ids of the lane's ad and cross groups, all in flight together
    id_t idv[NS];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      const int g = 4 * k + q;
      idv[k] = 0;
      if (k < KS && g >= nu && g < M) {
        const int f = g - nu;
        const bool is_ad = f < n_ad;
        const int fa = is_ad ? f : (gpu_cross ? s_pair[f - n_ad] >> 16 : f - n_ad);
        const id_t *ids = static_cast<const id_t *>(is_ad || gpu_cross ? a.ad_ids : a.cross_ids);
        idv[k] = ids[(int64_t)fa * R + rr];
      }
    }
    // table rows and both chunks of every group (loads of absent rows read
    // row 0 of a table and are zeroed)
    uint4 raw[NS][2];
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      raw[k][0] = raw[k][1] = make_uint4(0, 0, 0, 0);
      if (k < KS) {
        const int g = 4 * k + q;
        uint64_t addr = 0;
        if (g < M) {
          if (g < nu) {
            if (!users_lds) addr = reinterpret_cast<uint64_t>(Uh + (rq * nu + g) * EPG);
            if (a.rows_out && row_ok)
              a.rows_out[(int64_t)g * R + r] = users_lds ? s_urow[(int64_t)g * Q + rq] : a.urow[rq * nu + g];
          } else {
            int32_t row;
            const int f = g - nu;
            if (gpu_cross && f >= n_ad) {
              // user x ad cross value: key = mix64(user id) ^ ad id, hashed into
              // the group's table (ids as their unsigned bit patterns)
              const int fu = s_pair[f - n_ad] & 0xFFFF;
              const id_t *uids = static_cast<const id_t *>(a.user_ids);
              uint64_t uid, aid;
              if constexpr (HASHED) {
                uid = (uint64_t)uids[(int64_t)fu * Q + rq];
                aid = (uint64_t)idv[k];
              } else {
                uid = (uint64_t)(uint32_t)uids[(int64_t)fu * Q + rq];
                aid = (uint64_t)(uint32_t)idv[k];
              }
              const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
              row = (int32_t)mod_barrett(mix64((mix64(uid) ^ aid) ^ salt), (uint64_t)s_rows[g], s_magic[g]);
            } else if constexpr (HASHED) {
              const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
              row = (int32_t)mod_barrett(mix64((uint64_t)idv[k] ^ salt), (uint64_t)s_rows[g], s_magic[g]);
            } else {
              row = (int32_t)idv[k];
              if (row < 0 || row >= s_rows[g]) {
                atomicOr(a.err, 1);
                row = -1;
              }
            }
            if (a.rows_out && row_ok) a.rows_out[(int64_t)g * R + r] = row;
            if (row >= 0) addr = s_tab[g] + (uint64_t)row * (EPG * sizeof(TS));
          }
        }
        const uint64_t at = addr ? addr : dummy;
        const u32x4 v0 = *reinterpret_cast<gl_u32x4 *>(at);
        const u32x4 v1 = *reinterpret_cast<gl_u32x4 *>(at + 16);
        if (addr) {
          raw[k][0] = make_uint4(v0.x, v0.y, v0.z, v0.w);
          raw[k][1] = make_uint4(v1.x, v1.y, v1.z, v1.w);
        } else if (users_lds && g < nu) {
          raw[k][0] = s_uval[(rq * nu + g) * 2];
          raw[k][1] = s_uval[(rq * nu + g) * 2 + 1];
        }
      }
    }
    // squeeze and layer 1: h^T = ReLU(W1 z^T + b1)
    f32x4 h;
    {
      const float4 bv = s_b1[q];
      h[0] = bv.x; h[1] = bv.y; h[2] = bv.z; h[3] = bv.w;
    }
#pragma unroll
    for (int u = 0; u < NS / 4; ++u) {
      if (4 * u < KS) {
        const float4 wv = s_w1[u * 64 + lane];
        const float w[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int k = 4 * u + e;
          float v[EPG];
          Elem<TS>::unpack(raw[k][0], v);
          Elem<TS>::unpack(raw[k][1], v + EPC);
          float zs = 0.0f;
#pragma unroll
          for (int i = 0; i < EPG; ++i) zs += v[i];
          h = __builtin_amdgcn_mfma_f32_16x16x4f32(w[e], zs * inv_d, h, 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = h[e] > 0.0f ? h[e] : 0.0f;
    // layer 2: the weight of slot 4 gb + e in element e of block gb
    float sw[NS];
#pragma unroll
    for (int gb = 0; gb < NS / 4; ++gb) {
      if (gb < GB) {
        const float4 bv = s_b2[4 * gb + q], wv = s_w2[gb * 64 + lane];
        const float w[4] = {wv.x, wv.y, wv.z, wv.w};
        f32x4 o;
        o[0] = bv.x; o[1] = bv.y; o[2] = bv.z; o[3] = bv.w;
#pragma unroll
        for (int e = 0; e < 4; ++e) o = __builtin_amdgcn_mfma_f32_16x16x4f32(w[e], h[e], o, 0, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) sw[4 * gb + e] = 1.0f / (1.0f + expf(-o[e]));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) sw[4 * gb + e] = 0.0f;
      }
    }
    // reweight, linear_log, round once, store the group's two chunks
    if (row_ok) {
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        const int g = 4 * k + q;
        if (k < KS && g < M) {
          float v[EPG], o[EPG];
          Elem<TS>::unpack(raw[k][0], v);
          Elem<TS>::unpack(raw[k][1], v + EPC);
#pragma unroll
          for (int e = 0; e < EPG; ++e) {
            const float x = sw[k] * v[e];
            o[e] = LL ? linear_log(x) : x;
          }
          uint4 *dst = reinterpret_cast<uint4 *>(X + (r * M + g) * EPG);
          dst[0] = Elem<TS>::pack(o);
          dst[1] = Elem<TS>::pack(o + EPC);
          if (a.s_buf) a.s_buf[r * M + g] = sw[k];
        }
      }
    }
  }
}

template <typename TS, bool LL, int NS, bool ULDS>
static hipError_t gather_full_u(bool hashed, const GatherArgs &a, hipStream_t s) {
  const void *k = hashed ? reinterpret_cast<const void *>(&gather_full_kernel<TS, LL, true, NS, ULDS>)
                         : reinterpret_cast<const void *>(&gather_full_kernel<TS, LL, false, NS, ULDS>);
  const size_t shmem = ULDS ? (size_t)a.Q * a.n_user * 36 : 0;
  const int resident = resident_blocks(k, shmem);
  int64_t nb = ((a.R + 15) / 16 + 3) / 4;
  if (resident > 0 && nb > resident) nb = resident;
  if (hashed)
    hipLaunchKernelGGL((gather_full_kernel<TS, LL, true, NS, ULDS>), dim3((unsigned)nb), dim3(256), shmem, s, a);
  else
    hipLaunchKernelGGL((gather_full_kernel<TS, LL, false, NS, ULDS>), dim3((unsigned)nb), dim3(256), shmem, s, a);
  return hipGetLastError();
}

// One wave per 16 groups (models of 49 to 64 groups)
template <typename TS, bool LL, bool HASHED, bool ULDS>
__global__ __launch_bounds__(256) void gather_full_split_kernel(GatherArgs a) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;
  typedef typename std::conditional<HASHED, uint64_t, int32_t>::type id_t;
  constexpr int EPC = Elem<TS>::kPerChunk;   // elements per 16-byte chunk
  constexpr int EPG = 2 * EPC;               // elements per group (d)
  __shared__ uint64_t s_tab[kFullMaxM];
  __shared__ uint64_t s_magic[kFullMaxM];
  __shared__ int32_t s_rows[kFullMaxM];
  __shared__ int32_t s_pair[kFullMaxM];
  __shared__ int32_t s_req[kGatherMaxReqLds + 1];
  __shared__ float4 s_w1[kSeFullFloats / 4], s_w2[kSeFullFloats / 4];   // packed SE operands
  __shared__ float4 s_b1[4], s_b2[16];   // b1[4 q + e]; b2[16 gb + 4 e + q] at [4 gb + q].e
  __shared__ float4 s_hp[2][kFullMaxM / 16][64];   // the waves' layer-1 partial sums, by tile parity
  extern __shared__ __align__(16) unsigned char s_users[];   // [Q][nu][2] chunks, then [nu][Q] rows
  const int M = a.M, H = a.H, nu = a.n_user, n_ad = a.n_ad;
  const int64_t R = a.R, Q = a.Q;
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nt = blockDim.x, GB = nt >> 6;   // one wave per 16 groups
  for (int g = tid; g < M; g += nt) {
    s_tab[g] = reinterpret_cast<uint64_t>(a.tables[g]);
    s_magic[g] = a.table_magic[g];
    s_rows[g] = (int32_t)a.table_rows[g];
  }
  const bool gpu_cross = a.cross_pairs != nullptr;
  if (gpu_cross)
    for (int f = tid; f < a.n_cross; f += nt) s_pair[f] = a.cross_pairs[2 * f] | (a.cross_pairs[2 * f + 1] << 16);
  const bool req_in_lds = Q <= kGatherMaxReqLds;
  if (req_in_lds)
    for (int64_t i = tid; i <= Q; i += nt) s_req[i] = a.req_off[i];
  for (int i = tid; i < kSeFullFloats / 4; i += nt) {
    s_w1[i] = reinterpret_cast<const float4 *>(a.w1f)[i];
    s_w2[i] = reinterpret_cast<const float4 *>(a.w2f)[i];
  }
  if (tid < 16) {
    const int j = tid;
    reinterpret_cast<float *>(s_b1)[j] = j < H ? a.b1[j] : 0.0f;
  }
  if (tid < 64) {
    const int gb = tid >> 4, qq = (tid >> 2) & 3, e = tid & 3, g = 16 * gb + 4 * e + qq;
    reinterpret_cast<float *>(s_b2)[tid] = g < M ? a.b2[g] : 0.0f;
  }
  // few requests: their users' rows resolved and staged here (no pooling pass)
  uint4 *s_uval = reinterpret_cast<uint4 *>(s_users);
  int32_t *s_urow = reinterpret_cast<int32_t *>(s_users + (size_t)Q * nu * 32);
  if (ULDS) {
    for (int64_t i = tid; i < Q * nu * 2; i += nt) {
      const int p = (int)(i & 1);
      const int64_t qq = (i >> 1) / nu;
      const int f = (int)((i >> 1) - qq * nu);
      const int32_t row = resolve_row<HASHED>(a.user_ids, (int64_t)f * Q + qq, f, a.table_rows[f],
                                              a.table_magic[f], a.err);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0) v = reinterpret_cast<const uint4 *>(static_cast<const TS *>(a.tables[f]) + (int64_t)row * EPG)[p];
      s_uval[i] = v;
      if (p == 0) s_urow[(int64_t)f * Q + qq] = row;
    }
    // request offsets sanity (the pooling pass checks them otherwise)
    for (int64_t qq = (int64_t)blockIdx.x * nt + tid; qq < Q; qq += (int64_t)gridDim.x * nt) {
      bool bad = a.req_off[qq + 1] < a.req_off[qq];
      if (qq == 0) bad |= a.req_off[0] != 0;
      if (qq == Q - 1) bad |= (int64_t)a.req_off[Q] != R;
      if (bad) atomicOr(a.err, 2);
    }
  }
  __syncthreads();

  const float inv_d = 1.0f / (float)EPG;             // exact: EPG is a power of two
  const TS *Uh = static_cast<const TS *>(a.Uh);
  TS *X = static_cast<TS *>(a.X);
  const uint64_t dummy = s_tab[0];                   // row 0 of a table: always present
  const float4 w1v = s_w1[wave * 64 + lane], w2v = s_w2[wave * 64 + lane];
  const float4 b2v = s_b2[4 * wave + q];
  const float4 b1v = wave == 0 ? s_b1[q] : make_float4(0.f, 0.f, 0.f, 0.f);
  const float w1s[4] = {w1v.x, w1v.y, w1v.z, w1v.w}, w2s[4] = {w2v.x, w2v.y, w2v.z, w2v.w};

  const int64_t n_tiles = (R + 15) >> 4;
  int parity = 0;
  for (int64_t wt = blockIdx.x; wt < n_tiles; wt += gridDim.x, parity ^= 1) {
    const int64_t r = wt * 16 + c;
    const bool row_ok = r < R;
    const int64_t rr = row_ok ? r : R - 1;           // clamped: loaded, never stored
    int64_t rq = 0;
    if (nu > 0 || gpu_cross)
      rq = req_in_lds ? request_of_row(s_req, Q, rr) : request_of_row(a.req_off, Q, rr);

    // ids of the lane's ad and cross groups, all in flight together
    id_t idv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int g = 16 * wave + 4 * j + q;
      idv[j] = 0;
      if (g >= nu && g < M) {
        const int f = g - nu;
        const bool is_ad = f < n_ad;
        const int fa = is_ad ? f : (gpu_cross ? s_pair[f - n_ad] >> 16 : f - n_ad);
        const id_t *ids = static_cast<const id_t *>(is_ad || gpu_cross ? a.ad_ids : a.cross_ids);
        idv[j] = ids[(int64_t)fa * R + rr];
      }
    }
    // table rows and both chunks of every group (loads of absent rows read
    // row 0 of a table and are zeroed)
    uint4 raw[4][2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      raw[j][0] = raw[j][1] = make_uint4(0, 0, 0, 0);
      const int g = 16 * wave + 4 * j + q;
      uint64_t addr = 0;
      if (g < M) {
        if (g < nu) {
          if (!ULDS) addr = reinterpret_cast<uint64_t>(Uh + (rq * nu + g) * EPG);
          if (a.rows_out && row_ok)
            a.rows_out[(int64_t)g * R + r] = ULDS ? s_urow[(int64_t)g * Q + rq] : a.urow[rq * nu + g];
        } else {
          int32_t row;
          const int f = g - nu;
          if (gpu_cross && f >= n_ad) {
            // user x ad cross value: key = mix64(user id) ^ ad id, hashed into
            // the group's table (ids as their unsigned bit patterns)
            const int fu = s_pair[f - n_ad] & 0xFFFF;
            const id_t *uids = static_cast<const id_t *>(a.user_ids);
            uint64_t uid, aid;
            if constexpr (HASHED) {
              uid = (uint64_t)uids[(int64_t)fu * Q + rq];
              aid = (uint64_t)idv[j];
            } else {
              uid = (uint64_t)(uint32_t)uids[(int64_t)fu * Q + rq];
              aid = (uint64_t)(uint32_t)idv[j];
            }
            const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
            row = (int32_t)mod_barrett(mix64((mix64(uid) ^ aid) ^ salt), (uint64_t)s_rows[g], s_magic[g]);
          } else if constexpr (HASHED) {
            const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
            row = (int32_t)mod_barrett(mix64((uint64_t)idv[j] ^ salt), (uint64_t)s_rows[g], s_magic[g]);
          } else {
            row = (int32_t)idv[j];
            if (row < 0 || row >= s_rows[g]) {
              atomicOr(a.err, 1);
              row = -1;
            }
          }
          if (a.rows_out && row_ok) a.rows_out[(int64_t)g * R + r] = row;
          if (row >= 0) addr = s_tab[g] + (uint64_t)row * (EPG * sizeof(TS));
        }
      }
      const uint64_t at = addr ? addr : dummy;
      const u32x4 v0 = *reinterpret_cast<gl_u32x4 *>(at);
      const u32x4 v1 = *reinterpret_cast<gl_u32x4 *>(at + 16);
      if (addr) {
        raw[j][0] = make_uint4(v0.x, v0.y, v0.z, v0.w);
        raw[j][1] = make_uint4(v1.x, v1.y, v1.z, v1.w);
      } else if (ULDS && g < nu) {
        raw[j][0] = s_uval[(rq * nu + g) * 2];
        raw[j][1] = s_uval[(rq * nu + g) * 2 + 1];
      }
    }
    // squeeze and this wave's part of layer 1 (wave 0's part starts at b1)
    f32x4 hp;
    hp[0] = b1v.x; hp[1] = b1v.y; hp[2] = b1v.z; hp[3] = b1v.w;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v[EPG];
      Elem<TS>::unpack(raw[j][0], v);
      Elem<TS>::unpack(raw[j][1], v + EPC);
      float zs = 0.0f;
#pragma unroll
      for (int e = 0; e < EPG; ++e) zs += v[e];
      hp = __builtin_amdgcn_mfma_f32_16x16x4f32(w1s[j], zs * inv_d, hp, 0, 0, 0);
    }
    s_hp[parity][wave][lane] = make_float4(hp[0], hp[1], hp[2], hp[3]);
    __syncthreads();   // every wave's part is in; the other parity's buffer is free
    // h^T = ReLU(the parts in wave order), then layer 2 for block gb = wave
    f32x4 h;
    {
      float4 t = s_hp[parity][0][lane];
      h[0] = t.x; h[1] = t.y; h[2] = t.z; h[3] = t.w;
      for (int w = 1; w < GB; ++w) {
        t = s_hp[parity][w][lane];
        h[0] += t.x; h[1] += t.y; h[2] += t.z; h[3] += t.w;
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = h[e] > 0.0f ? h[e] : 0.0f;
    f32x4 o;
    o[0] = b2v.x; o[1] = b2v.y; o[2] = b2v.z; o[3] = b2v.w;
#pragma unroll
    for (int e = 0; e < 4; ++e) o = __builtin_amdgcn_mfma_f32_16x16x4f32(w2s[e], h[e], o, 0, 0, 0);
    // reweight, linear_log, round once, store the group's two chunks
    if (row_ok) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int g = 16 * wave + 4 * j + q;
        if (g < M) {
          const float sw = 1.0f / (1.0f + expf(-o[j]));
          float v[EPG], out[EPG];
          Elem<TS>::unpack(raw[j][0], v);
          Elem<TS>::unpack(raw[j][1], v + EPC);
#pragma unroll
          for (int e = 0; e < EPG; ++e) {
            const float x = sw * v[e];
            out[e] = LL ? linear_log(x) : x;
          }
          uint4 *dst = reinterpret_cast<uint4 *>(X + (r * M + g) * EPG);
          dst[0] = Elem<TS>::pack(out);
          dst[1] = Elem<TS>::pack(out + EPC);
          if (a.s_buf) a.s_buf[r * M + g] = sw;
        }
      }
    }
  }
}

template <typename TS, bool LL, bool ULDS>
static hipError_t gather_full_split_u(bool hashed, const GatherArgs &a, hipStream_t s) {
  const void *k = hashed ? reinterpret_cast<const void *>(&gather_full_split_kernel<TS, LL, true, ULDS>)
                         : reinterpret_cast<const void *>(&gather_full_split_kernel<TS, LL, false, ULDS>);
  const size_t shmem = ULDS ? (size_t)a.Q * a.n_user * 36 : 0;
  const int threads = 64 * ((a.M + 15) / 16);
  int per_cu = 0, dev = 0, cus = device_cus();
  if (hipGetDevice(&dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, threads, shmem) != hipSuccess)
    per_cu = 0;
  int64_t nb = (a.R + 15) / 16;
  if (per_cu > 0 && cus > 0 && nb > (int64_t)per_cu * cus) nb = (int64_t)per_cu * cus;
  if (hashed)
    hipLaunchKernelGGL((gather_full_split_kernel<TS, LL, true, ULDS>), dim3((unsigned)nb), dim3(threads), shmem, s, a);
  else
    hipLaunchKernelGGL((gather_full_split_kernel<TS, LL, false, ULDS>), dim3((unsigned)nb), dim3(threads), shmem, s, a);
  return hipGetLastError();
}

// Batches of few tiles, up to 48 groups: the one-wave form's arithmetic on
// one wave per 16 groups of a tile (wave w: slots 4 w .. 4 w + 3, groups
// 16 w + 4 j + q), so that a tile's gather, squeeze, reweighting and stores
// spread over GB = ceil(M / 16) waves. Layer 1's MFMA steps keep the one-wave
// order: wave w takes steps 4 w .. 4 w + 3 on the running sums that wave
// w - 1 left in LDS (wave 0 starts from b1), and the last wave's sums are
// every wave's h; layer 2's block w and the weights of the wave's slots are
// then the one-wave form's, bit for bit. Each wave keeps its groups' table
// pointers and SE operands in registers, and the first tile's ids and rows
// are fetched before the workgroup's set-up barrier, so their latency
// overlaps the users' resolution.
template <typename TS, bool LL, bool HASHED, bool ULDS>
__global__ __launch_bounds__(64 * (kFullTileM / 16)) void gather_full_chain_kernel(GatherArgs a) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(1))) const u32x4 gl_u32x4;
  typedef typename std::conditional<HASHED, uint64_t, int32_t>::type id_t;
  constexpr int EPC = Elem<TS>::kPerChunk;   // elements per 16-byte chunk
  constexpr int EPG = 2 * EPC;               // elements per group (d)
  __shared__ int32_t s_pair[kFullMaxM];
  __shared__ int32_t s_req[kGatherMaxReqLds + 1];
  __shared__ float4 s_h[2][kFullTileM / 16][64];   // layer-1 sums after wave w's steps, by tile parity
  extern __shared__ __align__(16) unsigned char s_users[];   // [Q][nu][2] chunks, then [nu][Q] rows
  const int M = a.M, H = a.H, nu = a.n_user, n_ad = a.n_ad;
  const int64_t R = a.R, Q = a.Q;
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nt = blockDim.x, GB = nt >> 6;   // one wave per 16 groups
  const bool gpu_cross = a.cross_pairs != nullptr;
  const int64_t n_tiles = (R + 15) >> 4;
  const float inv_d = 1.0f / (float)EPG;     // exact: EPG is a power of two
  const TS *Uh = static_cast<const TS *>(a.Uh);
  TS *X = static_cast<TS *>(a.X);
  uint4 *s_uval = reinterpret_cast<uint4 *>(s_users);
  int32_t *s_urow = reinterpret_cast<int32_t *>(s_users + (size_t)Q * nu * 32);

  // this lane's groups: table, row count and divisor magic
  const uint64_t dummy = reinterpret_cast<uint64_t>(a.tables[0]);   // row 0 of a table: always present
  uint64_t tab[4], magic[4];
  int32_t nrows[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int g = 16 * wave + 4 * j + q;
    const int gg = g < M ? g : 0;
    tab[j] = reinterpret_cast<uint64_t>(a.tables[gg]);
    magic[j] = a.table_magic[gg];
    nrows[j] = (int32_t)a.table_rows[gg];
  }
  // the wave's SE operands: b1[4 q + e]; W1, W2 and b2 of block gb = wave
  const float4 w1v = reinterpret_cast<const float4 *>(a.w1f)[wave * 64 + lane];
  const float4 w2v = reinterpret_cast<const float4 *>(a.w2f)[wave * 64 + lane];
  const float w1s[4] = {w1v.x, w1v.y, w1v.z, w1v.w}, w2s[4] = {w2v.x, w2v.y, w2v.z, w2v.w};
  float b1v[4], b2v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    b1v[e] = 4 * q + e < H ? a.b1[4 * q + e] : 0.0f;
    const int g2 = 16 * wave + 4 * e + q;
    b2v[e] = g2 < M ? a.b2[g2] : 0.0f;
  }

  // ids, table rows and both chunks of the tile's ad and cross groups (and
  // of the user groups from the pooling pass); loads of absent rows read row
  // 0 of a table and are zeroed
  id_t idv[4];
  uint4 raw[4][2];
  auto fetch = [&](int64_t wt, int64_t rq) {
    const int64_t r = wt * 16 + c;
    const bool row_ok = r < R;
    const int64_t rr = row_ok ? r : R - 1;   // clamped: loaded, never stored
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int g = 16 * wave + 4 * j + q;
      idv[j] = 0;
      if (g >= nu && g < M) {
        const int f = g - nu;
        const bool is_ad = f < n_ad;
        const int fa = is_ad ? f : (gpu_cross ? s_pair[f - n_ad] >> 16 : f - n_ad);
        const id_t *ids = static_cast<const id_t *>(is_ad || gpu_cross ? a.ad_ids : a.cross_ids);
        idv[j] = ids[(int64_t)fa * R + rr];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      raw[j][0] = raw[j][1] = make_uint4(0, 0, 0, 0);
      const int g = 16 * wave + 4 * j + q;
      uint64_t addr = 0;
      if (g < M) {
        if (g < nu) {
          if (!ULDS) {
            addr = reinterpret_cast<uint64_t>(Uh + (rq * nu + g) * EPG);
            if (a.rows_out && row_ok) a.rows_out[(int64_t)g * R + r] = a.urow[rq * nu + g];
          }
        } else {
          int32_t row;
          const int f = g - nu;
          if (gpu_cross && f >= n_ad) {
            // user x ad cross value: key = mix64(user id) ^ ad id, hashed into
            // the group's table (ids as their unsigned bit patterns)
            const int fu = s_pair[f - n_ad] & 0xFFFF;
            const id_t *uids = static_cast<const id_t *>(a.user_ids);
            uint64_t uid, aid;
            if constexpr (HASHED) {
              uid = (uint64_t)uids[(int64_t)fu * Q + rq];
              aid = (uint64_t)idv[j];
            } else {
              uid = (uint64_t)(uint32_t)uids[(int64_t)fu * Q + rq];
              aid = (uint64_t)(uint32_t)idv[j];
            }
            const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
            row = (int32_t)mod_barrett(mix64((mix64(uid) ^ aid) ^ salt), (uint64_t)nrows[j], magic[j]);
          } else if constexpr (HASHED) {
            const uint64_t salt = (uint64_t)(g + 1) * 0x9e3779b97f4a7c15ull;
            row = (int32_t)mod_barrett(mix64((uint64_t)idv[j] ^ salt), (uint64_t)nrows[j], magic[j]);
          } else {
            row = (int32_t)idv[j];
            if (row < 0 || row >= nrows[j]) {
              atomicOr(a.err, 1);
              row = -1;
            }
          }
          if (a.rows_out && row_ok) a.rows_out[(int64_t)g * R + r] = row;
          if (row >= 0) addr = tab[j] + (uint64_t)row * (EPG * sizeof(TS));
        }
      }
      if (g < M && (g >= nu || !ULDS)) {
        const uint64_t at = addr ? addr : dummy;
        const u32x4 v0 = *reinterpret_cast<gl_u32x4 *>(at);
        const u32x4 v1 = *reinterpret_cast<gl_u32x4 *>(at + 16);
        if (addr) {
          raw[j][0] = make_uint4(v0.x, v0.y, v0.z, v0.w);
          raw[j][1] = make_uint4(v1.x, v1.y, v1.z, v1.w);
        }
      }
    }
  };

  // the first tile's fetch needs no LDS unless user rows or cross pairs enter
  // it (request of a row from the LDS offsets)
  const bool hoist = !gpu_cross && (ULDS || nu == 0);
  int64_t wt = blockIdx.x;
  if (hoist && wt < n_tiles) fetch(wt, 0);

  if (gpu_cross)
    for (int f = tid; f < a.n_cross; f += nt) s_pair[f] = a.cross_pairs[2 * f] | (a.cross_pairs[2 * f + 1] << 16);
  const bool req_in_lds = Q <= kGatherMaxReqLds;
  if (req_in_lds)
    for (int64_t i = tid; i <= Q; i += nt) s_req[i] = a.req_off[i];
  // few requests: their users' rows resolved and staged here (no pooling pass)
  if (ULDS) {
    for (int64_t i = tid; i < Q * nu * 2; i += nt) {
      const int p = (int)(i & 1);
      const int64_t qq = (i >> 1) / nu;
      const int f = (int)((i >> 1) - qq * nu);
      const int32_t row = resolve_row<HASHED>(a.user_ids, (int64_t)f * Q + qq, f, a.table_rows[f],
                                              a.table_magic[f], a.err);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row >= 0) v = reinterpret_cast<const uint4 *>(static_cast<const TS *>(a.tables[f]) + (int64_t)row * EPG)[p];
      s_uval[i] = v;
      if (p == 0) s_urow[(int64_t)f * Q + qq] = row;
    }
    // request offsets sanity (the pooling pass checks them otherwise)
    for (int64_t qq = (int64_t)blockIdx.x * nt + tid; qq < Q; qq += (int64_t)gridDim.x * nt) {
      bool bad = a.req_off[qq + 1] < a.req_off[qq];
      if (qq == 0) bad |= a.req_off[0] != 0;
      if (qq == Q - 1) bad |= (int64_t)a.req_off[Q] != R;
      if (bad) atomicOr(a.err, 2);
    }
  }
  __syncthreads();

  int parity = 0;
  for (bool first = true; wt < n_tiles; wt += gridDim.x, parity ^= 1, first = false) {
    const int64_t r = wt * 16 + c;
    const bool row_ok = r < R;
    const int64_t rr = row_ok ? r : R - 1;
    int64_t rq = 0;
    if (nu > 0 || gpu_cross)
      rq = req_in_lds ? request_of_row(s_req, Q, rr) : request_of_row(a.req_off, Q, rr);
    if (!(hoist && first)) fetch(wt, rq);
    if (ULDS) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int g = 16 * wave + 4 * j + q;
        if (g < nu) {
          raw[j][0] = s_uval[(rq * nu + g) * 2];
          raw[j][1] = s_uval[(rq * nu + g) * 2 + 1];
          if (a.rows_out && row_ok) a.rows_out[(int64_t)g * R + r] = s_urow[(int64_t)g * Q + rq];
        }
      }
    }
    // squeeze of the wave's slots
    float zs[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float v[EPG];
      Elem<TS>::unpack(raw[j][0], v);
      Elem<TS>::unpack(raw[j][1], v + EPC);
      float t = 0.0f;
#pragma unroll
      for (int e = 0; e < EPG; ++e) t += v[e];
      zs[j] = t;
    }
    // layer 1 in the one-wave step order, handed from wave to wave
    for (int t = 0; t < GB; ++t) {
      if (wave == t) {
        f32x4 hp;
        if (t == 0) {
          hp[0] = b1v[0]; hp[1] = b1v[1]; hp[2] = b1v[2]; hp[3] = b1v[3];
        } else {
          const float4 v = s_h[parity][t - 1][lane];
          hp[0] = v.x; hp[1] = v.y; hp[2] = v.z; hp[3] = v.w;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) hp = __builtin_amdgcn_mfma_f32_16x16x4f32(w1s[j], zs[j] * inv_d, hp, 0, 0, 0);
        s_h[parity][t][lane] = make_float4(hp[0], hp[1], hp[2], hp[3]);
      }
      __syncthreads();
    }
    f32x4 h;
    {
      const float4 v = s_h[parity][GB - 1][lane];
      h[0] = v.x; h[1] = v.y; h[2] = v.z; h[3] = v.w;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = h[e] > 0.0f ? h[e] : 0.0f;
    // layer 2, block gb = wave: the weight of slot 4 gb + e in element e
    f32x4 o;
    o[0] = b2v[0]; o[1] = b2v[1]; o[2] = b2v[2]; o[3] = b2v[3];
#pragma unroll
    for (int e = 0; e < 4; ++e) o = __builtin_amdgcn_mfma_f32_16x16x4f32(w2s[e], h[e], o, 0, 0, 0);
    // reweight, linear_log, round once, store the group's two chunks
    if (row_ok) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int g = 16 * wave + 4 * j + q;
        if (g < M) {
          const float sw = 1.0f / (1.0f + expf(-o[j]));
          float v[EPG], out[EPG];
          Elem<TS>::unpack(raw[j][0], v);
          Elem<TS>::unpack(raw[j][1], v + EPC);
#pragma unroll
          for (int e = 0; e < EPG; ++e) {
            const float x = sw * v[e];
            out[e] = LL ? linear_log(x) : x;
          }
          uint4 *dst = reinterpret_cast<uint4 *>(X + (r * M + g) * EPG);
          dst[0] = Elem<TS>::pack(out);
          dst[1] = Elem<TS>::pack(out + EPC);
          if (a.s_buf) a.s_buf[r * M + g] = sw;
        }
      }
    }
  }
}

template <typename TS, bool LL, bool ULDS>
static hipError_t gather_full_chain_u(bool hashed, const GatherArgs &a, hipStream_t s) {
  const size_t shmem = ULDS ? (size_t)a.Q * a.n_user * 36 : 0;
  const int threads = 64 * ((a.M + 15) / 16);
  const int64_t nb = (a.R + 15) / 16;   // one tile per workgroup (few tiles)
  if (hashed)
    hipLaunchKernelGGL((gather_full_chain_kernel<TS, LL, true, ULDS>), dim3((unsigned)nb), dim3(threads), shmem, s, a);
  else
    hipLaunchKernelGGL((gather_full_chain_kernel<TS, LL, false, ULDS>), dim3((unsigned)nb), dim3(threads), shmem, s, a);
  return hipGetLastError();
}

// batches of at most two 16-row tiles per CU take the chained form (the
// one-wave form at 1,000 tiles and more)
static bool gather_full_chained(int64_t R) {
  const int cus = device_cus() > 0 ? device_cus() : 256;
  return (R + 15) / 16 <= 2 * (int64_t)cus;
}

// users' rows in LDS when the pooling pass does not run; up to 48 groups
// one wave per tile (the chained form of it for few tiles), above that one
// wave per 16 groups
template <typename TS, bool LL>
static hipError_t gather_full_t(bool hashed, const GatherArgs &a, hipStream_t s) {
  const bool pool = user_pool_needed(std::is_same<TS, float>::value ? kF32 : kBF16, a);
  if (a.M <= kFullTileM) {
    if (gather_full_chained(a.R))
      return pool ? gather_full_chain_u<TS, LL, false>(hashed, a, s)
                  : gather_full_chain_u<TS, LL, true>(hashed, a, s);
    return pool ? gather_full_u<TS, LL, kFullTileM / 4, false>(hashed, a, s)
                : gather_full_u<TS, LL, kFullTileM / 4, true>(hashed, a, s);
  }
  return pool ? gather_full_split_u<TS, LL, false>(hashed, a, s)
              : gather_full_split_u<TS, LL, true>(hashed, a, s);
}

hipError_t launch_gather_full(int dtype, bool linear_log, bool hashed, const GatherArgs &a,
                              hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  if (!gather_full_supported(dtype, a)) return hipErrorInvalidValue;
  switch (dtype) {
    case kF32: return linear_log ? gather_full_t<float, true>(hashed, a, s) : gather_full_t<float, false>(hashed, a, s);
    case kBF16: return linear_log ? gather_full_t<__bf16, true>(hashed, a, s) : gather_full_t<__bf16, false>(hashed, a, s);
    default: return linear_log ? gather_full_t<_Float16, true>(hashed, a, s) : gather_full_t<_Float16, false>(hashed, a, s);
  }
}

template <typename TS, int MODE, bool LL, int CPT, bool SE_LDS>
static hipError_t gather_se_l(bool hashed, const GatherArgs &a, int64_t blocks_needed, size_t shmem,
                              hipStream_t s) {
  const void *k = hashed ? reinterpret_cast<const void *>(&gather_se_kernel<TS, MODE, LL, true, CPT, SE_LDS>)
                         : reinterpret_cast<const void *>(&gather_se_kernel<TS, MODE, LL, false, CPT, SE_LDS>);
  const int resident = resident_blocks(k, shmem);
  int64_t nb = blocks_needed;
  if (resident > 0 && nb > resident) nb = resident;
  const dim3 grid((unsigned)nb);
  if (hashed)
    hipLaunchKernelGGL((gather_se_kernel<TS, MODE, LL, true, CPT, SE_LDS>), grid, dim3(kGatherThreads),
                       shmem, s, a);
  else
    hipLaunchKernelGGL((gather_se_kernel<TS, MODE, LL, false, CPT, SE_LDS>), grid, dim3(kGatherThreads),
                       shmem, s, a);
  return hipGetLastError();
}

template <typename TS, int MODE, bool LL, int CPT>
static hipError_t gather_se_c(bool hashed, GatherArgs a, hipStream_t s) {
  constexpr int EPC = Elem<TS>::kPerChunk;
  const int nax = a.n_ad + a.n_cross;
  const int cpr = a.M * (a.d / EPC);
  // rows per wave: as many as the chunk budget allows, fewer for small
  // batches so that about 2048 waves are launched (one 2,000-ad request:
  // one row per wave)
  const int t_max = (64 * CPT) / cpr;
  const int64_t t_fill = (a.R + 2047) / 2048;
  const int T = t_fill < t_max ? (t_fill < 1 ? 1 : (int)t_fill) : t_max;
  a.rows_per_tile = T;
  a.Mp = (a.M + 3) & ~3;
  a.Hp = (a.H + 3) & ~3;
  a.mg_tw = div_magic((uint32_t)T);
  a.mg_h = div_magic((uint32_t)a.H);
  a.mg_m = div_magic((uint32_t)a.M);
  a.mg_ns = div_magic((uint32_t)(a.n_seq > 0 ? a.n_seq : 1));
  a.mg_sd4 = div_magic((uint32_t)(a.n_seq > 0 ? a.n_seq * a.d / 4 : 1));
  a.wave_lds_bytes = (int32_t)((sizeof(float) * (size_t)T * (a.Mp + a.Hp + a.n_seq * a.d + a.M) +
                                sizeof(int32_t) * (size_t)(T * nax + T) + 15) / 16 * 16);
  a.meta_lds_bytes = (int32_t)((24 * (size_t)a.M + 15) / 16 * 16);
  a.req_lds_bytes = a.Q + 1 <= kGatherMaxReqLds ? (int32_t)((4 * (a.Q + 1) + 15) / 16 * 16) : 0;
  a.users_in_lds = user_pool_needed(std::is_same<TS, float>::value ? kF32 : kBF16, a) ? 0 : 1;
  a.urow_lds_bytes = a.users_in_lds ? (int32_t)((4 * (int64_t)a.n_user * a.Q + 15) / 16 * 16) : 0;
  a.uval_lds_bytes = a.users_in_lds ? (int32_t)((int64_t)a.n_user * a.Q * a.d * sizeof(TS)) : 0;
  const size_t se_floats = (size_t)a.H * a.Mp + (size_t)a.M * a.Hp + a.H + a.M;
  a.se_in_lds = (MODE == kFull || MODE == kWeightsOnly) && se_floats * sizeof(float) <= 24 * 1024;
  a.se_lds_bytes = a.se_in_lds ? (int32_t)((se_floats * sizeof(float) + 15) / 16 * 16) : 0;
  const size_t shmem = (size_t)a.meta_lds_bytes + a.req_lds_bytes + a.urow_lds_bytes +
                       a.uval_lds_bytes + a.se_lds_bytes + 4 * (size_t)a.wave_lds_bytes;
  if (T * nax > 64 * kGatherMaxIdsPerLane || shmem > 160 * 1024) return hipErrorInvalidValue;
  const int64_t rows_per_block = 4 * (int64_t)T;
  const int64_t blocks = (a.R + rows_per_block - 1) / rows_per_block;
  if (a.se_in_lds) return gather_se_l<TS, MODE, LL, CPT, true>(hashed, a, blocks, shmem, s);
  return gather_se_l<TS, MODE, LL, CPT, false>(hashed, a, blocks, shmem, s);
}

// chunks per lane: 8 (a wave holds 512 / chunks-per-row rows); 16 only when a
// row has more than 512 chunks
template <typename TS, int MODE, bool LL>
static hipError_t gather_se_t(bool hashed, const GatherArgs &a, hipStream_t s) {
  const int cpr = a.M * (a.d / Elem<TS>::kPerChunk);
  if (cpr > 512) return gather_se_c<TS, MODE, LL, 16>(hashed, a, s);
  return gather_se_c<TS, MODE, LL, 8>(hashed, a, s);
}

template <typename TS>
static hipError_t gather_se_dt(int mode, bool ll, bool hashed, const GatherArgs &a, hipStream_t s) {
  if (mode == kWeightsOnly) return gather_se_t<TS, kWeightsOnly, false>(hashed, a, s);
  if (mode == kSqueezeRaw) {
    if (a.n_seq > 0 || !a.z_out) return hipErrorInvalidValue;   // pooled sums are not exact in TS
    return gather_se_t<TS, kSqueezeRaw, false>(hashed, a, s);
  }
  if (mode == kRawOut) return gather_se_t<TS, kRawOut, false>(hashed, a, s);
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
  if (n_parts % kSelQuarters != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mask_select_kernel, dim3((unsigned)Q), dim3(1024),
                     sizeof(float) * (kSelQuarters + 1) * M, s, partial, req_off, R, M, n_parts, k,
                     mask, mask_out);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void transpose_f32_kernel(const float *__restrict__ src,
                                                            float *__restrict__ dst, int32_t rows,
                                                            int32_t cols) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)rows * cols) return;
  const int32_t r = (int32_t)(i / cols), c = (int32_t)(i - (int64_t)r * cols);
  dst[(int64_t)c * rows + r] = src[i];
}

hipError_t launch_transpose_f32(const float *src, float *dst, int32_t rows, int32_t cols,
                                hipStream_t s) {
  const int64_t n = (int64_t)rows * cols;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(transpose_f32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src,
                     dst, rows, cols);
  return hipGetLastError();
}

// ------------------------------------------------------------- se_rows
// SE weights of rows from their squeeze (Eq. 2 read as squeeze -> FC ->
// ReLU -> FC -> sigmoid), for models whose SE parameters do not fit the
// gather's LDS budget, on the fp32 matrix cores.  A workgroup takes 16 rows
// at a time and forms both layers transposed,
//   h^T [H x 16] = ReLU(W1 [H x M] z^T [M x 16] + b1),
//   s^T [M x 16] = sigmoid(W2 [M x H] h^T [H x 16] + b2),
// as 16x16x4 fp32 MFMAs, so that layer 1's output fragments are layer 2's B
// operand without a transpose.  Wave w owns hidden units 16w .. 16w + 15 in
// layer 1 and output blocks w, w + 4, ... in layer 2; lane l (row or unit
// l % 16, quarter q = l / 16) feeds K index q * MQ + t at step t of layer 1
// and hidden unit 4 t + q at step t of layer 2.  Both weight matrices are
// packed once at load time in that operand order (one 16-byte vector per lane
// and 4 steps, zero past M and H), held in registers for all of the
// workgroup's rows; the rows' squeeze is staged in LDS with coalesced loads.
// Products and sums are fp32; the sums run in the matrix cores' order
// instead of index order, which only moves fp32 rounding.
constexpr int kSeTile = 16;
constexpr int kSeMaxH = 64;     // four 16-wide hidden blocks, one per wave
constexpr int kSeMaxGB = 16;    // M <= 256: 16-wide output blocks, four per wave

__host__ __device__ static int se_rows_mq(int M) { return ((M + 3) / 4 + 3) & ~3; }   // K run of a quarter, % 4 == 0
static int se_rows_nc(int M) {                                    // 4-step chunks the kernel holds
  const int mq = se_rows_mq(M);
  return mq <= 16 ? 4 : mq <= 32 ? 8 : 16;
}

void se_rows_packed_floats(int32_t M, int32_t H, size_t *n1, size_t *n2) {
  const bool ok = M > 0 && M <= 256 && H > 0 && H <= kSeMaxH;
  *n1 = ok ? (size_t)(kSeMaxH / 16) * se_rows_nc(M) * 256 : 0;
  *n2 = ok ? (size_t)((M + 15) / 16) * 4 * 256 : 0;
}

// one thread per packed word: W1p [4 hidden blocks][NC chunks][64 lanes][4],
// then W2p [output blocks][4 chunks][64 lanes][4]
__global__ __launch_bounds__(256) void pack_se_rows_kernel(const float *__restrict__ w1,
                                                           const float *__restrict__ w2, int M,
                                                           int H, int MQ, int NC,
                                                           float *__restrict__ w1p,
                                                           float *__restrict__ w2p, int64_t n1,
                                                           int64_t n2) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int e = (int)(i & 3), lane = (int)((i >> 2) & 63), c = lane & 15, q = lane >> 4;
  if (i < n1) {
    const int u = (int)((i >> 8) % NC), b = (int)((i >> 8) / NC);
    const int j = 16 * b + c, k = 4 * u + e, g = q * MQ + k;
    w1p[i] = j < H && k < MQ && g < M ? w1[(int64_t)j * M + g] : 0.0f;
  } else if (i < n1 + n2) {
    const int64_t i2 = i - n1;
    const int v = (int)((i2 >> 8) & 3), gb = (int)(i2 >> 10);
    const int g = 16 * gb + c, jj = 4 * (4 * v + e) + q;
    w2p[i2] = g < M && jj < H ? w2[(int64_t)g * H + jj] : 0.0f;
  }
}

hipError_t launch_pack_se_rows(const float *w1, const float *w2, int32_t M, int32_t H, float *w1p,
                               float *w2p, hipStream_t s) {
  size_t n1, n2;
  se_rows_packed_floats(M, H, &n1, &n2);
  if (n1 == 0) return hipErrorInvalidValue;
  const int64_t n = (int64_t)(n1 + n2);
  hipLaunchKernelGGL(pack_se_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, w1, w2,
                     M, H, se_rows_mq(M), se_rows_nc(M), w1p, w2p, (int64_t)n1, (int64_t)n2);
  return hipGetLastError();
}

template <int NC>
__global__ __launch_bounds__(256) void se_rows_kernel(const float *__restrict__ z,
                                                      float *__restrict__ s_out, int64_t R, int M,
                                                      int H, const float4 *__restrict__ w1p,
                                                      const float *__restrict__ b1,
                                                      const float4 *__restrict__ w2p,
                                                      const float *__restrict__ b2,
                                                      float *__restrict__ tpart) {
  constexpr int kMaxStride = 16 * NC + 4;
  __shared__ __align__(16) float zs[kSeTile * kMaxStride];   // row c at c * ZST
  __shared__ float hs[kSeMaxH * kSeTile];                     // h^T: unit j, row c at j * 16 + c
  const int tid = threadIdx.x, lane = tid & 63, c = lane & 15, q = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int MQ = se_rows_mq(M), MP = 4 * MQ;   // padded row: zeros from M to MP
  const int ZST = MP + 4;                      // an odd number of 16-byte slots: no bank conflicts
  const int GB = (M + 15) >> 4;
  float4 wa[NC], wb[kSeMaxGB / 4][4];
#pragma unroll
  for (int u = 0; u < NC; ++u) wa[u] = w1p[(wave * NC + u) * 64 + lane];
#pragma unroll
  for (int i = 0; i < kSeMaxGB / 4; ++i) {
    const int gb = wave + 4 * i;
#pragma unroll
    for (int v = 0; v < 4; ++v)
      wb[i][v] = gb < GB ? w2p[(gb * 4 + v) * 64 + lane] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float bias1[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int jj = wave * 16 + 4 * q + e;
    bias1[e] = jj < H ? b1[jj] : 0.0f;
  }
  for (int64_t r0 = (int64_t)blockIdx.x * kSeTile; r0 < R; r0 += (int64_t)gridDim.x * kSeTile) {
    // the tile's squeeze rows (contiguous in z) into LDS; rows past R and
    // columns past M are zeros
    {
      const int rows = R - r0 < kSeTile ? (int)(R - r0) : kSeTile;
      const float *zt = z + r0 * M;
      float v[kSeTile];
#pragma unroll
      for (int cc = 0; cc < kSeTile; ++cc)
        v[cc] = tid < M && cc < rows ? zt[cc * M + tid] : 0.0f;
#pragma unroll
      for (int cc = 0; cc < kSeTile; ++cc)
        if (tid < MP) zs[cc * ZST + tid] = v[cc];
    }
    __syncthreads();
    // layer 1
    f32x4 acc;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = bias1[e];
    const float *zrow = zs + c * ZST + q * MQ;
#pragma unroll
    for (int u = 0; u < NC; ++u) {
      if (4 * u < MQ) {
        const float4 zv = *reinterpret_cast<const float4 *>(zrow + 4 * u);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u].x, zv.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u].y, zv.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u].z, zv.z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u].w, zv.w, acc, 0, 0, 0);
      }
    }
    // lane holds h[row r0 + c][unit wave * 16 + 4 q + e]; padded units are 0
#pragma unroll
    for (int e = 0; e < 4; ++e)
      hs[(wave * 16 + 4 * q + e) * kSeTile + c] = acc[e] > 0.0f ? acc[e] : 0.0f;
    __syncthreads();
    // layer 2
    float hb[kSeMaxH / 4];
#pragma unroll
    for (int t = 0; t < kSeMaxH / 4; ++t) hb[t] = hs[(4 * t + q) * kSeTile + c];
    const int64_t row = r0 + c;
#pragma unroll
    for (int i = 0; i < kSeMaxGB / 4; ++i) {
      const int gb = wave + 4 * i;
      if (gb < GB) {
        f32x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int gg = gb * 16 + 4 * q + e;
          o[e] = gg < M ? b2[gg] : 0.0f;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          o = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[i][v].x, hb[4 * v], o, 0, 0, 0);
          o = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[i][v].y, hb[4 * v + 1], o, 0, 0, 0);
          o = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[i][v].z, hb[4 * v + 2], o, 0, 0, 0);
          o = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[i][v].w, hb[4 * v + 3], o, 0, 0, 0);
        }
        // lane holds s[row r0 + c][group gb * 16 + 4 q + e]
        float sv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) sv[e] = 1.0f / (1.0f + expf(-o[e]));
        if (row < R) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int gg = gb * 16 + 4 * q + e;
            if (gg < M) s_out[row * M + gg] = sv[e];
          }
        }
        if (tpart) {
          // the tile's sum of each group's weight over its rows: a fixed
          // butterfly over the 16 lanes of a quarter, lane c = 0 stores it
#pragma unroll
          for (int e = 0; e < 4; ++e) sv[e] = row < R ? sv[e] : 0.0f;
#pragma unroll
          for (int off = 1; off < 16; off <<= 1)
#pragma unroll
            for (int e = 0; e < 4; ++e) sv[e] += __shfl_xor(sv[e], off);
          if (c == 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int gg = gb * 16 + 4 * q + e;
              if (gg < M) tpart[(r0 / kSeTile) * M + gg] = sv[e];
            }
          }
        }
      }
    }
    // the next tile's staging writes only zs, which no wave reads after its
    // layer 1; hs is written again only after the next barrier
  }
}

hipError_t launch_se_rows(const float *z, float *s_out, int64_t R, int32_t M, int32_t H,
                          const float *w1p, const float *b1, const float *w2p, const float *b2,
                          float *tile_part, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (M <= 0 || M > 256 || H <= 0 || H > kSeMaxH) return hipErrorInvalidValue;
  if ((reinterpret_cast<uintptr_t>(w1p) | reinterpret_cast<uintptr_t>(w2p)) & 15)
    return hipErrorInvalidValue;
  const int cus = device_cus();
  if (cus <= 0) return hipErrorInvalidValue;
  const int64_t tiles = (R + kSeTile - 1) / kSeTile;
  const unsigned grid = (unsigned)(tiles < 2 * cus ? tiles : 2 * cus);
  const float4 *a1 = reinterpret_cast<const float4 *>(w1p);
  const float4 *a2 = reinterpret_cast<const float4 *>(w2p);
  switch (se_rows_nc(M)) {
    case 4: hipLaunchKernelGGL(se_rows_kernel<4>, dim3(grid), dim3(256), 0, s, z, s_out, R, M, H, a1, b1, a2, b2, tile_part); break;
    case 8: hipLaunchKernelGGL(se_rows_kernel<8>, dim3(grid), dim3(256), 0, s, z, s_out, R, M, H, a1, b1, a2, b2, tile_part); break;
    default: hipLaunchKernelGGL(se_rows_kernel<16>, dim3(grid), dim3(256), 0, s, z, s_out, R, M, H, a1, b1, a2, b2, tile_part);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------- apply_weights
// The network input in place from the gathered rows: each 16-byte chunk of
// row r, group g becomes round(LL(s[r][g] e)) for a group the request keeps
// and 0 for one its mask drops (Section 3.2 reweighting, Eq. 3 when LL).
// A workgroup takes kApplyRows rows and finds their requests once, in LDS;
// each thread loads all of its chunks and weights before it computes.
constexpr int kApplyRows = 2;
constexpr int kApplyPerThread = 4;
template <typename TS, bool LL>
__global__ __launch_bounds__(256) void apply_weights_kernel(TS *__restrict__ X,
                                                            const float *__restrict__ s_buf,
                                                            const uint8_t *__restrict__ mask,
                                                            const int32_t *__restrict__ req_off,
                                                            int64_t Q, int64_t R, int M, int lcpg,
                                                            int CPR, uint32_t mg_cpr) {
  constexpr int EPC = Elem<TS>::kPerChunk;
  __shared__ int32_t s_rq[kApplyRows];
  const int64_t r0 = (int64_t)blockIdx.x * kApplyRows;
  const int rows = R - r0 < kApplyRows ? (int)(R - r0) : kApplyRows;
  if (threadIdx.x < rows) s_rq[threadIdx.x] = (int32_t)request_of_row(req_off, Q, r0 + threadIdx.x);
  __syncthreads();
  uint4 *xc = reinterpret_cast<uint4 *>(X) + r0 * CPR;
  const int n = rows * CPR;
  for (int base = 0; base < n; base += 256 * kApplyPerThread) {
    uint4 raw[kApplyPerThread];
    float sg[kApplyPerThread];
    bool keep[kApplyPerThread];
#pragma unroll
    for (int u = 0; u < kApplyPerThread; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      raw[u] = make_uint4(0, 0, 0, 0);
      sg[u] = 0.0f;
      keep[u] = false;
      if (idx < n) {
        const int t = fast_div(idx, mg_cpr), g = (idx - t * CPR) >> lcpg;
        raw[u] = xc[idx];
        sg[u] = s_buf[(r0 + t) * M + g];
        keep[u] = !mask || mask[(int64_t)s_rq[t] * M + g] != 0;
      }
    }
#pragma unroll
    for (int u = 0; u < kApplyPerThread; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      if (idx < n) {
        float v[EPC], o[EPC];
        Elem<TS>::unpack(raw[u], v);
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
          const float x = sg[u] * v[e];
          o[e] = keep[u] ? (LL ? linear_log(x) : x) : 0.0f;
        }
        xc[idx] = Elem<TS>::pack(o);
      }
    }
  }
}

template <typename TS>
static hipError_t apply_t(bool ll, void *X, const float *s_buf, const uint8_t *mask,
                          const int32_t *req_off, int64_t Q, int64_t R, int32_t M, int32_t d,
                          hipStream_t s) {
  constexpr int EPC = Elem<TS>::kPerChunk;
  const int cpg = d / EPC, cpr = M * cpg;
  if (cpg <= 0 || (cpg & (cpg - 1)) || kApplyRows * (int64_t)cpr >= (1 << 16)) return hipErrorInvalidValue;
  const int lcpg = __builtin_ctz(cpg);
  const dim3 grid((unsigned)((R + kApplyRows - 1) / kApplyRows));
  if (ll)
    hipLaunchKernelGGL((apply_weights_kernel<TS, true>), grid, dim3(256), 0, s, static_cast<TS *>(X),
                       s_buf, mask, req_off, Q, R, M, lcpg, cpr, div_magic((uint32_t)cpr));
  else
    hipLaunchKernelGGL((apply_weights_kernel<TS, false>), grid, dim3(256), 0, s, static_cast<TS *>(X),
                       s_buf, mask, req_off, Q, R, M, lcpg, cpr, div_magic((uint32_t)cpr));
  return hipGetLastError();
}

// ------------------------------------------------------------- apply_compact
// The network input of a model whose requests keep k of the M groups, with
// the dropped groups left out instead of zeroed (Section 3.2 feature group
// selection): row r of request q holds, in group order, the kp = min(k, M)
// groups that q keeps (kept[q][j]), each 16-byte chunk round(LL(s[r][g] e))
// of the gathered row (Eq. 3 when LL). The gathered rows stay in place; the
// compacted rows go to Xc [R][kp * d]. A workgroup takes kApplyRows rows and
// finds their requests and kept lists once, in LDS. The grid's next Q * N
// workgroups copy, for request q, row n of the first layer's weights W
// [N][M * d] restricted to the kept groups into Wc [Q][N][kp * d] (the
// first layer's operand for that request), and its last one lays out the
// first layer's row tiles (build_row_tiles) for the tile height that layer
// uses.
template <typename TS, bool LL>
__global__ __launch_bounds__(256) void apply_compact_kernel(const TS *__restrict__ Xraw,
                                                            TS *__restrict__ Xc,
                                                            const float *__restrict__ s_buf,
                                                            const int32_t *__restrict__ kept,
                                                            const int32_t *__restrict__ req_off,
                                                            int64_t Q, int64_t R, int M, int kp,
                                                            int lcpg, int CPR, int CPRC,
                                                            uint32_t mg_cprc, int64_t n_apply,
                                                            const uint4 *__restrict__ W, int64_t N,
                                                            uint4 *__restrict__ Wc, int BR, int64_t cap,
                                                            RowTile *__restrict__ tiles,
                                                            int32_t *__restrict__ n_tiles) {
  constexpr int EPC = Elem<TS>::kPerChunk;
  __shared__ int32_t s_rq[kApplyRows];
  __shared__ int32_t s_kept[kApplyRows][256];
  __shared__ int64_t s_scan[256];
  if ((int64_t)blockIdx.x >= n_apply) {
    const int64_t wrow = (int64_t)blockIdx.x - n_apply;
    if (wrow == Q * N) {
      build_row_tiles<256>(req_off, Q, R, BR, cap, tiles, n_tiles, s_scan);
      return;
    }
    const int64_t q = wrow / N, n = wrow - q * N;
    const int32_t *kq = kept + q * kp;
    const uint4 *src = W + n * CPR;
    uint4 *dst = Wc + wrow * CPRC;
    for (int c = threadIdx.x; c < CPRC; c += 256) {
      const int j = c >> lcpg, h = c & ((1 << lcpg) - 1);
      int g = kq[j];
      g = g < 0 ? 0 : (g < M ? g : M - 1);
      dst[c] = src[(g << lcpg) + h];
    }
    return;
  }
  const int64_t r0 = (int64_t)blockIdx.x * kApplyRows;
  const int rows = R - r0 < kApplyRows ? (int)(R - r0) : kApplyRows;
  if (threadIdx.x < rows) s_rq[threadIdx.x] = (int32_t)request_of_row(req_off, Q, r0 + threadIdx.x);
  __syncthreads();
  for (int i = threadIdx.x; i < rows * kp; i += 256) {
    const int t = i / kp, j = i - t * kp;
    s_kept[t][j] = kept[(int64_t)s_rq[t] * kp + j];
  }
  __syncthreads();
  const uint4 *xr = reinterpret_cast<const uint4 *>(Xraw) + r0 * CPR;
  uint4 *xc = reinterpret_cast<uint4 *>(Xc) + r0 * CPRC;
  const int n = rows * CPRC;
  for (int base = 0; base < n; base += 256 * kApplyPerThread) {
    uint4 raw[kApplyPerThread];
    float sg[kApplyPerThread];
#pragma unroll
    for (int u = 0; u < kApplyPerThread; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      raw[u] = make_uint4(0, 0, 0, 0);
      sg[u] = 0.0f;
      if (idx < n) {
        const int t = fast_div(idx, mg_cprc), c = idx - t * CPRC;
        const int j = c >> lcpg, h = c & ((1 << lcpg) - 1);
        int g = s_kept[t][j];
        g = g < 0 ? 0 : (g < M ? g : M - 1);
        raw[u] = xr[(int64_t)t * CPR + (g << lcpg) + h];
        sg[u] = s_buf[(r0 + t) * M + g];
      }
    }
#pragma unroll
    for (int u = 0; u < kApplyPerThread; ++u) {
      const int idx = base + u * 256 + threadIdx.x;
      if (idx < n) {
        float v[EPC], o[EPC];
        Elem<TS>::unpack(raw[u], v);
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
          const float x = sg[u] * v[e];
          o[e] = LL ? linear_log(x) : x;
        }
        xc[idx] = Elem<TS>::pack(o);
      }
    }
  }
}

template <typename TS>
static hipError_t apply_compact_t(bool ll, const void *Xraw, void *Xc, const float *s_buf,
                                  const int32_t *kept, const int32_t *req_off, int64_t Q,
                                  int64_t R, int32_t M, int32_t kp, int32_t d, const void *W,
                                  int32_t N, void *Wc, RowTile *tiles, int32_t *n_tiles,
                                  hipStream_t s) {
  constexpr int EPC = Elem<TS>::kPerChunk;
  const int cpg = d / EPC, cpr = M * cpg, cprc = kp * cpg;
  if (cpg <= 0 || (cpg & (cpg - 1)) || kp <= 0 || kp > M || M > 256 || N <= 0 || Q <= 0 ||
      kApplyRows * (int64_t)cpr >= (1 << 16) || !dense_grouped_supported(
          std::is_same<TS, float>::value ? kF32 : kBF16, N, kp * d))
    return hipErrorInvalidValue;
  const int lcpg = __builtin_ctz(cpg);
  const int64_t n_apply = (R + kApplyRows - 1) / kApplyRows;
  const int64_t blocks = n_apply + Q * (int64_t)N + 1;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  const int BR = dense_grouped_tile_rows(R, N, kp * d);
  const int64_t cap = row_tiles_bound(R, Q, BR);
  const dim3 grid((unsigned)blocks);
  if (ll)
    hipLaunchKernelGGL((apply_compact_kernel<TS, true>), grid, dim3(256), 0, s,
                       static_cast<const TS *>(Xraw), static_cast<TS *>(Xc), s_buf, kept, req_off,
                       Q, R, M, kp, lcpg, cpr, cprc, div_magic((uint32_t)cprc), n_apply,
                       static_cast<const uint4 *>(W), (int64_t)N, static_cast<uint4 *>(Wc), BR, cap,
                       tiles, n_tiles);
  else
    hipLaunchKernelGGL((apply_compact_kernel<TS, false>), grid, dim3(256), 0, s,
                       static_cast<const TS *>(Xraw), static_cast<TS *>(Xc), s_buf, kept, req_off,
                       Q, R, M, kp, lcpg, cpr, cprc, div_magic((uint32_t)cprc), n_apply,
                       static_cast<const uint4 *>(W), (int64_t)N, static_cast<uint4 *>(Wc), BR, cap,
                       tiles, n_tiles);
  return hipGetLastError();
}

hipError_t launch_apply_compact(int dtype, bool ll, const void *Xraw, void *Xc, const float *s_buf,
                                const int32_t *kept, const int32_t *req_off, int64_t Q, int64_t R,
                                int32_t M, int32_t kp, int32_t d, const void *W, int32_t N,
                                void *Wc, RowTile *tiles, int32_t *n_tiles, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  switch (dtype) {
    case kBF16: return apply_compact_t<__bf16>(ll, Xraw, Xc, s_buf, kept, req_off, Q, R, M, kp, d, W, N, Wc, tiles, n_tiles, s);
    case kF16: return apply_compact_t<_Float16>(ll, Xraw, Xc, s_buf, kept, req_off, Q, R, M, kp, d, W, N, Wc, tiles, n_tiles, s);
    default: return hipErrorInvalidValue;   // the grouped first layer is bf16 or fp16
  }
}

hipError_t launch_apply_weights(int dtype, bool ll, void *X, const float *s_buf,
                                const uint8_t *mask, const int32_t *req_off, int64_t Q, int64_t R,
                                int32_t M, int32_t d, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  switch (dtype) {
    case kF32: return apply_t<float>(ll, X, s_buf, mask, req_off, Q, R, M, d, s);
    case kBF16: return apply_t<__bf16>(ll, X, s_buf, mask, req_off, Q, R, M, d, s);
    default: return apply_t<_Float16>(ll, X, s_buf, mask, req_off, Q, R, M, d, s);
  }
}

hipError_t launch_clear_flag(int32_t *err, hipStream_t s) {
  hipLaunchKernelGGL(clear_flag_kernel, dim3(1), dim3(1), 0, s, err);
  return hipGetLastError();
}

}  // namespace cold
