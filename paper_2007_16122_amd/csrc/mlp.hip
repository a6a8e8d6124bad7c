// mlp.hip -- the fully connected network of the COLD model (Section 4.1:
// D_in x 1024 x 512 x 256 x 128 x 64 x 2) on gfx950.
//
//  dense_relu_buf   Y = ReLU(X W^T + b) for bf16/fp16 X, W with fp32
//                   accumulation on the matrix cores
//                   (v_mfma_f32_16x16x32_{bf16,f16}) and one rounding of the
//                   output to the storage type.  Operand tiles stream from
//                   global memory straight into an LDS ring (no VGPR staging);
//                   W plays the MFMA A operand (output features on the rows),
//                   X the B operand.  Tiles are numbered so that the
//                   workgroups sharing one row block of X run on the same XCD
//                   (workgroup i is dispatched to XCD i mod 8) and reuse it
//                   from that XCD's L2.  256 x 256 tiles (8 waves) for large
//                   batches, 64 x 64 for a single request.
//  dense_relu_mfma  the same layer with register-staged, double-buffered LDS
//                   tiles; used when K is not a multiple of 32.
//  dense_tail       the last separate hidden layer (512 -> 256) fused with
//                   the tail: the last two hidden layers and the head, with
//                   the tail's activations carried at about twice the
//                   storage precision (hi/lo pairs, see the tail section).
//  mlp_tail         the tail alone over 64-row tiles held in LDS.
//  dense_relu_f32   the layer in fp32 FMA (the fp32 model).
//  head             last layer (n_out = 1 or 2) in fp32 plus sigmoid or
//                   two-way softmax; writes the CTR.
#include <type_traits>

#include "cold_internal.h"

namespace cold {

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

// Block tile BR rows x BN output features, 4 waves as 2 x 2, each wave
// (BR/2) x (BN/2).  Per 32-deep K step a wave reads BR/32 + BN/32 fragments
// of 16 bytes per lane and issues (BR/32)*(BN/32) MFMAs.
template <typename TS, int BR, int BN>
__global__ __launch_bounds__(256, 2) void dense_relu_mfma_kernel(const TS *__restrict__ X,
                                                                 const TS *__restrict__ W,
                                                                 const float *__restrict__ bias,
                                                                 TS *__restrict__ Y, int64_t R, int N,
                                                                 int K, int tiles_n, int tiles_total) {
  typedef typename Mfma<TS>::frag frag;
  constexpr int NI = BN / 32;              // 16-wide feature blocks per wave
  constexpr int RJ = BR / 32;              // 16-wide row blocks per wave
  constexpr int A_PER_T = BN * kBK / 8 / 256;   // 16-byte chunks of the W tile per thread
  constexpr int B_PER_T = BR * kBK / 8 / 256;
  static_assert(A_PER_T >= 1 && B_PER_T >= 1, "tile/thread mismatch");

  __shared__ __align__(16) TS sA[2][BN * kLdsRow];
  __shared__ __align__(16) TS sB[2][BR * kLdsRow];

  const int tile = xcd_tile(blockIdx.x, tiles_total);
  const int tr = tile / tiles_n, tn = tile - tr * tiles_n;
  const int64_t r0 = (int64_t)tr * BR;
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
    frag fa[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i)
      fa[i] = *reinterpret_cast<const frag *>(&sA[buf][(wn * (BN / 2) + i * 16 + frow) * kLdsRow + fk]);
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
      const frag fb = *reinterpret_cast<const frag *>(&sB[buf][(wr * (BR / 2) + j * 16 + frow) * kLdsRow + fk]);
#pragma unroll
      for (int i = 0; i < NI; ++i) acc[i][j] = Mfma<TS>::mac(fa[i], fb, acc[i][j]);
    }
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
      const int64_t r = r0 + wr * (BR / 2) + j * 16 + dr;
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

// ---------------------------------------------------------------------------
// Pipelined layer, dense_relu_buf: operand tiles stream global -> LDS with the
// gfx950 buffer loads to LDS (each lane's 16 bytes land at base + 16 * lane,
// no VGPR staging) into an S-stage ring, issued S-1 K steps ahead; each wave
// waits only for its own loads of the stage it is about to read (vmcnt), then
// one barrier per K step.  LDS rows are 64 bytes (32 elements); chunk c of
// row r sits in slot c ^ swz(r), which makes the 16-byte fragment reads
// conflict-free whether the LDS serves 8 or 16 lanes per cycle.  The output
// tile is staged in LDS after the K loop so every row segment is written with
// full 16-byte stores.
__device__ __forceinline__ int lds_swz(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
// the same for 128-byte rows (64-deep K steps): rows r and r + 1 are 128 bytes
// apart, so the eight 16-byte slots of rows r & 7 are permuted by r & 7 and the
// two halves of a 16-row block by one more bit
__device__ __forceinline__ int lds_swz64(int r) { return (r & 7) ^ ((r >> 3) & 1); }


// wait until at most min(later, MAXL) stages of LOADS loads each are in flight
template <int LOADS, int MAXL>
__device__ __forceinline__ void wait_stages(int later) {
  if constexpr (MAXL > 0) {
    if (later >= MAXL) {
      wait_vm<MAXL * LOADS>();
      return;
    }
    wait_stages<LOADS, MAXL - 1>(later);
  } else {
    wait_vm<0>();
  }
}

// The instruction stream of the K loop is kept lean:
//  * one buffer resource per operand starts at the tile's first row; a lane
//    has a fixed offset and the K step is a scalar offset, so a K step costs
//    no vector address arithmetic; rows past the end of the operand read
//    zeros (the resource's range check);
//  * the wave index is uniform, so every LDS destination is scalar;
//  * the K loop is unrolled over the ring, so every LDS read address is a
//    compile-time offset from one register;
//  * the accumulators start at the bias;
//  * the epilogue rounds two outputs per instruction and applies ReLU to the
//    rounded pair as 16-bit integers (round-to-nearest-even is monotone and
//    keeps 0, and a negative half-precision value has its sign bit set, so
//    max(bits, 0) as signed integers is ReLU after rounding).
// Waves are laid out 2 (rows) x WN (features); each wave owns a
// (BR/2) x (BN/WN) block of 16 x 16 MFMA tiles.
template <typename TS> struct Pair;
template <> struct Pair<__bf16> {
  typedef __bf16 v2 __attribute__((ext_vector_type(2)));
};
template <> struct Pair<_Float16> {
  typedef _Float16 v2 __attribute__((ext_vector_type(2)));
};

// 16 bytes per lane from base + voff + soff into LDS at dst + 16 * lane;
// reads at or past base + bytes return zeros
__device__ __forceinline__ void buffer_load_lds16(const void *base, int bytes, void *dst, int voff,
                                                  int soff) {
  typedef __attribute__((address_space(3))) void lds_void;
  constexpr int kRsrcWord3 = 0x00020000;   // raw buffer, 32-bit data format
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes, kRsrcWord3);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)dst, 16, voff, soff, 0, 0);
}

__device__ __forceinline__ uint32_t relu_bits2(uint32_t v) {
  typedef short s2 __attribute__((ext_vector_type(2)));
  const s2 r = __builtin_elementwise_max(__builtin_bit_cast(s2, v), (s2){0, 0});
  return __builtin_bit_cast(uint32_t, r);
}

template <typename TS>
__device__ __forceinline__ uint32_t round2(float lo, float hi) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  const typename Pair<TS>::v2 h = __builtin_convertvector((f2){lo, hi}, typename Pair<TS>::v2);
  return __builtin_bit_cast(uint32_t, h);
}

// Tile geometry of the pipelined layer: BR x BN outputs over 2 x WN waves,
// KB-deep ring stages (32: 64-byte LDS rows; 64: 128-byte rows).
template <int BR, int BN, int S, int WN, int KB = 32> struct BufTile {
  static constexpr int NT = 128 * WN, NW = 2 * WN;          // threads, waves
  static constexpr int NI = BN / WN / 16, RJ = BR / 32;     // 16x16 blocks per wave
  static constexpr int ROWB = KB * 2;                       // bytes per LDS row
  static constexpr int CPRW = KB / 8;                       // 16-byte chunks per LDS row
  static constexpr int RPI = 64 / CPRW;                     // rows per load instruction
  static constexpr int STAGE = (BN + BR) * ROWB;            // bytes per ring stage
  static constexpr int LOADS = (BN + BR) / RPI / NW;        // loads per wave per stage
  static constexpr int RING = S * STAGE;
  static_assert(KB == 32 || KB == 64, "stage depth");
  static_assert((BN + BR) % (RPI * NW) == 0, "loads must split evenly over the waves");
  static_assert(BN % (16 * WN) == 0 && BR % 32 == 0 && BN % RPI == 0, "tile shape");
  static_assert(S >= 2 && S <= 4, "stages");
  static_assert(RJ >= 1, "row blocks");
};

// The K loop of one tile: acc[i][j] = bias + W X^T over K for the
// (wn, wr) wave's blocks; lane holds D[4*(lane/16) + e][lane % 16] of block
// (i, j), i.e. output features n0 + wn*(BN/WN) + 16 i + 4 (lane/16) + e of row
// r0 + wr*(BR/2) + 16 j + lane % 16.  smem holds the ring (RING bytes); on
// return the ring is free once the workgroup has passed a barrier.
template <typename TS, int BR, int BN, int S, int WN, int KB = 32, bool HALF = false>
__device__ __forceinline__ void buf_tile_kloop(
    const TS *__restrict__ X, const TS *__restrict__ W, const float *__restrict__ bias, int64_t R,
    int N, int K, int64_t r0, int n0, unsigned char *smem,
    f32x4 (&acc)[BufTile<BR, BN, S, WN, KB>::NI][BufTile<BR, BN, S, WN, KB>::RJ]) {
  typedef typename Mfma<TS>::frag frag;
  typedef BufTile<BR, BN, S, WN, KB> G;
  constexpr int NI = G::NI, RJ = G::RJ, ROWB = G::ROWB, STAGE = G::STAGE, LOADS = G::LOADS;
  constexpr int CPRW = G::CPRW, RPI = G::RPI;
  auto swz = [](int r) { return KB == 32 ? lds_swz(r) : lds_swz64(r); };
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wn = wave % WN, wr = wave / WN;

  // operand windows: W rows [n0, n0 + min(BN, N - n0)), X rows [r0, r0 + min(BR, R - r0))
  const int w_rows = N - n0 < BN ? N - n0 : BN;
  const int x_rows = R - r0 < BR ? (int)(R - r0) : BR;
  const TS *wbase = W + (int64_t)n0 * K, *xbase = X + r0 * K;
  const int wbytes = w_rows * K * 2, xbytes = x_rows * K * 2;

  // load instruction ins fills RPI consecutive LDS rows (W rows first, then
  // X rows); lane l writes slot l % CPRW of row l / CPRW, which holds the
  // row's logical chunk slot ^ swz(row)
  int voff[LOADS];
#pragma unroll
  for (int u = 0; u < LOADS; ++u) {
    const int ins = wave * LOADS + u;
    const int rin = lane / CPRW, slot = lane % CPRW;
    const int row = (ins < BN / RPI ? ins : ins - BN / RPI) * RPI + rin;
    const int chunk = slot ^ swz(row & 15);
    voff[u] = (row * K + chunk * 8) * 2;
  }
  auto issue = [&](int ks, int stage) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int ins = wave * LOADS + u;
      const bool is_w = ins < BN / RPI;
      const int dst = is_w ? ins * RPI * ROWB : BN * ROWB + (ins - BN / RPI) * RPI * ROWB;
      buffer_load_lds16(is_w ? static_cast<const void *>(wbase) : static_cast<const void *>(xbase),
                        is_w ? wbytes : xbytes, smem + stage * STAGE + dst, voff[u], ks * (KB * 2));
    }
  };

  // bias of this lane's output features (clamped; features past N are not
  // stored) becomes the accumulators' starting value
  const int dn = (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    f32x4 bv;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = n0 + wn * (BN / WN) + i * 16 + dn + e;
      bv[e] = bias[n < N ? n : N - 1];
    }
#pragma unroll
    for (int j = 0; j < RJ; ++j) acc[i][j] = bv;
  }

  // HALF (64-deep stages, K % 64 == 32): the last stage is a half stage;
  // its second 32 of K lie past the rows' ends and are loaded (the next
  // row's first elements, or zeros past the operand window) but not used,
  // so the sum still runs over the same 32-deep K blocks in the same order
  static_assert(!HALF || KB == 64, "half stages of 64-deep stages");
  const int ksteps = HALF ? (K + KB - 1) / KB : K / KB;
#pragma unroll
  for (int st = 0; st < S - 1; ++st)
    if (st < ksteps) issue(st, st);

  // fragment reads: 32-deep half h of a stage is logical chunks 4 h + lane / 16
  const int frow = lane & 15, fc = lane >> 4;
  int a_off[KB / 32], b_off[KB / 32];
#pragma unroll
  for (int h = 0; h < KB / 32; ++h) {
    const int pc = ((4 * h + fc) ^ swz(frow)) * 16;
    a_off[h] = (wn * (BN / WN) + frow) * ROWB + pc;
    b_off[h] = BN * ROWB + (wr * (BR / 2) + frow) * ROWB + pc;
  }
  for (int kb = 0; kb < ksteps; kb += S) {
#pragma unroll
    for (int st = 0; st < S; ++st) {
      const int ks = kb + st;
      if (ks < ksteps) {
        // stage ks must have landed: later stages issued so far = min(S-2, ksteps-1-ks)
        wait_stages<LOADS, S - 2>(ksteps - 1 - ks);
        compiler_fence();
        __builtin_amdgcn_s_barrier();
        compiler_fence();
        if (ks + S - 1 < ksteps) issue(ks + S - 1, (st + S - 1) % S);
        const unsigned char *base = smem + st * STAGE;
#pragma unroll
        for (int h = 0; h < KB / 32; ++h) {
          if constexpr (HALF)
            if (h > 0 && ks == ksteps - 1) break;   // the same for every wave
          frag fa[NI], fb[RJ];
#pragma unroll
          for (int i = 0; i < NI; ++i)
            fa[i] = *reinterpret_cast<const frag *>(base + a_off[h] + i * 16 * ROWB);
#pragma unroll
          for (int j = 0; j < RJ; ++j)
            fb[j] = *reinterpret_cast<const frag *>(base + b_off[h] + j * 16 * ROWB);
#pragma unroll
          for (int j = 0; j < RJ; ++j)
#pragma unroll
            for (int i = 0; i < NI; ++i) acc[i][j] = Mfma<TS>::mac(fa[i], fb[j], acc[i][j]);
          // issue order: the A fragments and two B fragments (one with a
          // single row block), then one B fragment read after each row
          // block's NI MFMAs, so that a read is two blocks ahead of the
          // MFMAs that use it
          constexpr int AHEAD = RJ < 2 ? RJ : 2;
          __builtin_amdgcn_sched_group_barrier(0x100, NI + AHEAD, 0);   // DS reads
#pragma unroll
          for (int j = 0; j < RJ - AHEAD; ++j) {
            __builtin_amdgcn_sched_group_barrier(0x008, NI, 0);         // MFMAs
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, AHEAD * NI, 0);
        }
      }
    }
  }
  wait_vm<0>();
}

// GRP: the rows belong to requests with weights of their own; row tile tr
// is entry tr of the device-built table (rows [r0, r0 + n) of request q,
// whose weights start w_stride elements after the previous request's), and
// workgroups past the table's count have no tile.
template <typename TS, int BR, int BN, int S, int WN = 2, int MINW = 2, int KB = 32, bool GRP = false,
          bool HALF = false>
__global__ __launch_bounds__(128 * WN, MINW) void dense_relu_buf_kernel(const TS *__restrict__ X,
                                                                     const TS *__restrict__ W,
                                                                     const float *__restrict__ bias,
                                                                     TS *__restrict__ Y, int64_t R,
                                                                     int N, int K, int tiles_n,
                                                                     int tiles_total,
                                                                     const RowTile *__restrict__ rtiles,
                                                                     const int32_t *__restrict__ n_rtiles,
                                                                     int64_t w_stride) {
  typedef BufTile<BR, BN, S, WN, KB> G;
  constexpr int NT = G::NT, NI = G::NI, RJ = G::RJ;
  constexpr int OUT_STRIDE = BN + 8;                 // elements per staged output row
  // the output tile is staged through the ring in one pass, or in two
  // passes of BR/2 rows when the whole tile does not fit
  constexpr int OUT_PASSES = BR * OUT_STRIDE * 2 <= G::RING ? 1 : 2;
  constexpr int OUT_BYTES = BR / OUT_PASSES * OUT_STRIDE * 2;
  constexpr int SMEM = G::RING > OUT_BYTES ? G::RING : OUT_BYTES;
  __shared__ __align__(16) unsigned char smem[SMEM];

  const int tile = xcd_tile(blockIdx.x, tiles_total);
  const int tr = tile / tiles_n, tn = tile - tr * tiles_n;
  int64_t r0 = (int64_t)tr * BR;
  const TS *Wt = W;
  if constexpr (GRP) {
    if (tr >= *n_rtiles) return;   // the same for the whole workgroup
    const RowTile t = rtiles[tr];
    r0 = t.r0;
    R = t.r0 + t.n;
    Wt = W + (int64_t)t.q * w_stride;
  }
  const int n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave % WN, wr = wave / WN;
  const int dn = (lane >> 4) * 4, dr = lane & 15;

  f32x4 acc[NI][RJ];
  buf_tile_kloop<TS, BR, BN, S, WN, KB, HALF>(X, Wt, bias, R, N, K, r0, n0, smem, acc);

  // epilogue: round, ReLU, stage the tile in LDS, write rows with 16-byte
  // stores.
  compiler_fence();
  __builtin_amdgcn_s_barrier();
  compiler_fence();
  uint16_t *sout = reinterpret_cast<uint16_t *>(smem);
  constexpr int PR = BR / OUT_PASSES;   // rows per pass
  constexpr int CPRW = BN / 8;          // 16-byte chunks per output row
#pragma unroll
  for (int pass = 0; pass < OUT_PASSES; ++pass) {
    if (OUT_PASSES == 1 || wr == pass) {
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int nl = wn * (BN / WN) + i * 16 + dn;
#pragma unroll
        for (int j = 0; j < RJ; ++j) {
          const int rl = (OUT_PASSES == 1 ? wr * (BR / 2) : 0) + j * 16 + dr;
          uint2 packed;
          packed.x = relu_bits2(round2<TS>(acc[i][j][0], acc[i][j][1]));
          packed.y = relu_bits2(round2<TS>(acc[i][j][2], acc[i][j][3]));
          *reinterpret_cast<uint2 *>(sout + rl * OUT_STRIDE + nl) = packed;
        }
      }
    }
    compiler_fence();
    __syncthreads();
    for (int idx = tid; idx < PR * CPRW; idx += NT) {
      const int rl = idx / CPRW, c = idx - rl * CPRW;
      const int64_t r = r0 + pass * PR + rl;
      const int n = n0 + c * 8;
      if (r < R && n < N)
        *reinterpret_cast<uint4 *>(Y + r * N + n) =
            *reinterpret_cast<const uint4 *>(sout + rl * OUT_STRIDE + c * 8);
    }
    if (pass + 1 < OUT_PASSES) {
      compiler_fence();
      __syncthreads();
    }
  }
}

// Fragment-major weights of the fused tail: a [N][K] matrix (N % 16 == 0,
// K % 32 == 0) stored as one 1 KB block per (16-feature block fb, 32-deep K
// step k), in MFMA operand order: lane l holds features fb*16 + l % 16, K
// elements 32 k + 8 (l / 16) .. + 8.  A wave then loads a fragment as one
// contiguous 1 KB block instead of 16 half-used cache lines.
__host__ __device__ inline int64_t frag_offset(int fb, int k, int ksteps, int lane) {
  return ((int64_t)(fb * ksteps + k) * 64 + lane) * 8;
}

// one 16-byte chunk per thread: row-major chunk (n, k..k+7) to its fragment-major place
__global__ __launch_bounds__(256) void pack_frag_kernel(const uint4 *__restrict__ src,
                                                        uint4 *__restrict__ dst, int64_t N, int32_t K) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t cpr = K / 8;
  if (c >= N * cpr) return;
  const int64_t n = c / cpr;
  const int k = (int)(c - n * cpr) * 8;
  const int lane = ((k & 31) >> 3) * 16 + (int)(n & 15);
  dst[frag_offset((int)(n >> 4), k >> 5, K / 32, lane) / 8] = src[c];
}

hipError_t launch_pack_frag(const void *src, void *dst, int64_t N, int32_t K, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (N % 16 != 0 || K % 32 != 0) return hipErrorInvalidValue;
  const int64_t chunks = N * (K / 8);
  hipLaunchKernelGGL(pack_frag_kernel, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s,
                     static_cast<const uint4 *>(src), static_cast<uint4 *>(dst), N, K);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fused tail: the last two hidden layers and the output head, K0 -> N1 -> N2
// (ReLU) -> n_out (sigmoid or softmax), on row tiles held in LDS; the small
// weight matrices (N1 x K0 and N2 x N1, fragment-major, see frag_offset) are
// read as MFMA fragments straight from global memory, where every workgroup
// finds them in L2.
//
// Precision of the tail. Its layers are narrow (the last one feeds the 64
// inputs of the head directly), so rounding their activations to the storage
// type moves the CTR more than the rounding of every wider layer before them.
// The tail therefore carries each hidden activation v (fp32, after bias and
// ReLU) as a pair hi = RNE(v), lo = RNE(v - hi) of storage-type values (v - hi
// is exact in fp32), about twice the storage precision, and a layer takes
// both halves through the matrix cores: W hi + W lo, two MFMAs per product,
// summed in fp32. The last hidden layer's output stays in fp32 and the head
// reads it as such. Every sum of the tail runs in the same order whichever
// kernel, tile shape or wave computes it.

// the two storage-type values packed in one 32-bit word, widened to fp32
template <typename TS> __device__ __forceinline__ void unpack2(uint32_t w, float &a, float &b);
template <> __device__ __forceinline__ void unpack2<__bf16>(uint32_t w, float &a, float &b) {
  a = __uint_as_float(w << 16);
  b = __uint_as_float(w & 0xFFFF0000u);
}
template <> __device__ __forceinline__ void unpack2<_Float16>(uint32_t w, float &a, float &b) {
  a = static_cast<float>(__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu)));
  b = static_cast<float>(__builtin_bit_cast(_Float16, (uint16_t)(w >> 16)));
}

// hi/lo pairs of two fp32 values (see above); a value whose hi is not finite
// (beyond the storage range) gets lo = 0
template <typename TS>
__device__ __forceinline__ void split2(float v0, float v1, uint32_t &hi, uint32_t &lo) {
  hi = round2<TS>(v0, v1);
  float h0, h1;
  unpack2<TS>(hi, h0, h1);
  const float d0 = __builtin_isfinite(h0) ? v0 - h0 : 0.0f;
  const float d1 = __builtin_isfinite(h1) ? v1 - h1 : 0.0f;
  lo = round2<TS>(d0, d1);
}

// MFMA sums of one tail layer on rows held in LDS: acc[i][j] = sum over K of
// W[n][k] in[r][k] for the 16-row blocks jb0 .. jb0 + JB - 1 and the
// NB 16-feature blocks of wf, from zero, K steps in order. in_at(row, c) is
// the LDS address of 16-byte chunk c of an input row; with EXT the low halves
// of the input sit lo_bytes after the high halves, and each K step adds
// W hi, then W lo. wf[k][i] is the weight fragment of feature block i and K
// step k.
template <typename TS, int KS, int NB, int JB, bool EXT, typename InAt>
__device__ __forceinline__ void tail_mma(const InAt &in_at, int lo_bytes,
                                         const typename Mfma<TS>::frag (&wf)[KS][NB], int jb0,
                                         int lane, f32x4 (&acc)[NB][JB]) {
  typedef typename Mfma<TS>::frag frag;
  const int frow = lane & 15, fq = lane >> 4;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < JB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < KS; ++k) {
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      const TS *p = in_at((jb0 + j) * 16 + frow, 4 * k + fq);
      const frag fb = *reinterpret_cast<const frag *>(p);
      frag fl;
      if constexpr (EXT) fl = *reinterpret_cast<const frag *>(reinterpret_cast<const char *>(p) + lo_bytes);
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        acc[i][j] = Mfma<TS>::mac(wf[k][i], fb, acc[i][j]);
        if constexpr (EXT) acc[i][j] = Mfma<TS>::mac(wf[k][i], fl, acc[i][j]);
      }
    }
  }
}

// bias, ReLU, then the hi/lo pair of every output: row (jb0 + j) * 16 + lane % 16,
// features (nb0 + i) * 16 + 4 (lane / 16) .. + 3; the low halves go lo_elems
// elements after the high halves
template <typename TS, int NB, int JB>
__device__ __forceinline__ void tail_store_ext(const f32x4 (&acc)[NB][JB], const float *__restrict__ bg,
                                               TS *out, int stride, int lo_elems, int nb0, int jb0,
                                               int lane) {
  const int dn = (lane >> 4) * 4, dr = lane & 15;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int n = (nb0 + i) * 16 + dn;
    float bv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) bv[e] = bg[n + e];
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float t = acc[i][j][e] + bv[e];
        v[e] = t > 0.0f ? t : 0.0f;
      }
      uint2 hi, lo;
      split2<TS>(v[0], v[1], hi.x, lo.x);
      split2<TS>(v[2], v[3], hi.y, lo.y);
      TS *o = out + ((jb0 + j) * 16 + dr) * stride + n;
      *reinterpret_cast<uint2 *>(o) = hi;
      *reinterpret_cast<uint2 *>(o + lo_elems) = lo;
    }
  }
}

// bias and ReLU in fp32, stored as fp32 (the last hidden layer)
template <int NB, int JB>
__device__ __forceinline__ void tail_store_f32(const f32x4 (&acc)[NB][JB], const float *__restrict__ bg,
                                               float *out, int stride, int nb0, int jb0, int lane) {
  const int dn = (lane >> 4) * 4, dr = lane & 15;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int n = (nb0 + i) * 16 + dn;
    float bv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) bv[e] = bg[n + e];
#pragma unroll
    for (int j = 0; j < JB; ++j) {
      float4 v;
      v.x = acc[i][j][0] + bv[0];
      v.y = acc[i][j][1] + bv[1];
      v.z = acc[i][j][2] + bv[2];
      v.w = acc[i][j][3] + bv[3];
      v.x = v.x > 0.0f ? v.x : 0.0f;
      v.y = v.y > 0.0f ? v.y : 0.0f;
      v.z = v.z > 0.0f ? v.z : 0.0f;
      v.w = v.w > 0.0f ? v.w : 0.0f;
      *reinterpret_cast<float4 *>(out + ((jb0 + j) * 16 + dr) * stride + n) = v;
    }
  }
}

// Output head of the fused tail on fp32 rows: 4 threads per row (row tid / 4),
// each summing a quarter of the N2 inputs in order, then two shuffle steps;
// sigmoid (one logit) or two-way softmax, CTR = class 1. row_of maps the
// LDS row to the batch row; rows at or past R are not stored.
template <int N2, typename RowOf>
__device__ __forceinline__ void tail_head(const float *h2, int s2, const float *s_wh,
                                          const float *s_bh, int n_out, float *__restrict__ scores,
                                          const RowOf &row_of, int64_t R, int tid) {
  const int row = tid >> 2, q = tid & 3;
  float z0 = 0.0f, z1 = 0.0f;
#pragma unroll 4
  for (int k = q * (N2 / 4); k < (q + 1) * (N2 / 4); ++k) {
    const float x = h2[row * s2 + k];
    z0 += s_wh[k] * x;
    if (n_out > 1) z1 += s_wh[N2 + k] * x;
  }
  z0 += __shfl_xor(z0, 1);
  z0 += __shfl_xor(z0, 2);
  z1 += __shfl_xor(z1, 1);
  z1 += __shfl_xor(z1, 2);
  const int64_t r = row_of(row);
  if (q == 0 && r < R) {
    z0 += s_bh[0];
    if (n_out > 1) z1 += s_bh[1];
    scores[r] = n_out == 1 ? 1.0f / (1.0f + expf(-z0)) : 1.0f / (1.0f + expf(z0 - z1));
  }
}

// The tail as a kernel of its own (the layer before it is not fused with
// it: its K is not a multiple of 64, or there is none): 64-row tiles, input
// tile in the storage type from global memory, first layer on it, then the
// extended-precision second layer and head. Two workgroups per CU (the
// second hidden tile takes the input tile's LDS once the first layer is done).
template <typename TS, int K0, int N1, int N2>
__global__ __launch_bounds__(256, 2) void mlp_tail_kernel(const TS *__restrict__ A,
                                                       const TS *__restrict__ W1,
                                                       const float *__restrict__ b1,
                                                       const TS *__restrict__ W2,
                                                       const float *__restrict__ b2,
                                                       const TS *__restrict__ Wh,
                                                       const float *__restrict__ bh, int n_out,
                                                       float *__restrict__ scores, int64_t R) {
  typedef typename Mfma<TS>::frag frag;
  constexpr int BR = 64;
  constexpr int S0 = K0 + 8, S1 = N1 + 8, S2 = N2 + 4;   // padded LDS rows
  static_assert(K0 % 32 == 0 && N1 % 32 == 0 && N2 % 32 == 0 && N1 % 64 == 0 && N2 % 64 == 0,
                "tail widths");
  static_assert(BR * S2 * 4 <= BR * S0 * 2, "the last hidden tile fits in the input tile");
  __shared__ __align__(16) TS s_in[BR * S0];
  __shared__ __align__(16) TS s_h1[2 * BR * S1];       // hi, then lo
  float *s_h2 = reinterpret_cast<float *>(s_in);        // after the first layer
  __shared__ float s_wh[2 * N2];
  __shared__ float s_bh[2];

  const int64_t r0 = (int64_t)blockIdx.x * BR;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // input tile (rows past the end are clamped: loaded, never stored); every
  // load is issued before the first LDS store so the tile costs one HBM
  // round trip, not one per chunk
  constexpr int CPR0 = K0 / 8, NLD = BR * CPR0 / 256;
  static_assert((BR * CPR0) % 256 == 0, "tile chunks");
  uint4 tile[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int c = tid + i * 256;
    const int row = c / CPR0, kc = c - row * CPR0;
    int64_t r = r0 + row;
    r = r < R ? r : R - 1;
    tile[i] = *reinterpret_cast<const uint4 *>(A + r * K0 + kc * 8);
  }

  // The weight fragments of both layers are loaded once, before the input
  // tile is needed, so their L2 latency overlaps the tile load instead of
  // stalling every K step.
  constexpr int NB1 = N1 / 4 / 16, KS1 = K0 / 32;   // layer 1: blocks per wave, K steps
  constexpr int NB2 = N2 / 4 / 16, KS2 = N1 / 32;   // layer 2
  frag w1f[KS1][NB1], w2f[KS2][NB2];
#pragma unroll
  for (int k = 0; k < KS1; ++k)
#pragma unroll
    for (int i = 0; i < NB1; ++i)
      w1f[k][i] = *reinterpret_cast<const frag *>(W1 + frag_offset(wave * NB1 + i, k, KS1, lane));
#pragma unroll
  for (int k = 0; k < KS2; ++k)
#pragma unroll
    for (int i = 0; i < NB2; ++i)
      w2f[k][i] = *reinterpret_cast<const frag *>(W2 + frag_offset(wave * NB2 + i, k, KS2, lane));
  static_assert(2 * N2 <= 256, "one head weight per thread");
  const TS whv = Wh[tid < n_out * N2 ? tid : 0];
  const float bhv = bh[tid < n_out ? tid : 0];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int c = tid + i * 256;
    const int row = c / CPR0, kc = c - row * CPR0;
    *reinterpret_cast<uint4 *>(&s_in[row * S0 + kc * 8]) = tile[i];
  }
  if (tid < n_out * N2) s_wh[tid] = Elem<TS>::to_f32(whv);
  if (tid < n_out) s_bh[tid] = bhv;
  __syncthreads();   // input tile and head weights in LDS

  // wave w owns the output features [w*N/4, (w+1)*N/4) of each layer
  auto in0 = [&](int row, int c) { return s_in + row * S0 + c * 8; };
  f32x4 a1[NB1][BR / 16];
  tail_mma<TS, KS1, NB1, BR / 16, false>(in0, 0, w1f, 0, lane, a1);
  tail_store_ext<TS, NB1, BR / 16>(a1, b1, s_h1, S1, BR * S1, wave * NB1, 0, lane);
  __syncthreads();   // the input tile is dead: the last hidden tile takes its place
  auto in1 = [&](int row, int c) { return s_h1 + row * S1 + c * 8; };
  f32x4 a2[NB2][BR / 16];
  tail_mma<TS, KS2, NB2, BR / 16, true>(in1, BR * S1 * 2, w2f, 0, lane, a2);
  tail_store_f32<NB2, BR / 16>(a2, b2, s_h2, S2, wave * NB2, 0, lane);
  __syncthreads();
  tail_head<N2>(s_h2, S2, s_wh, s_bh, n_out, scores, [&](int row) { return r0 + row; }, R, tid);
}

// The last separate hidden layer and the fused tail in one kernel, when that
// layer is 256 wide (the tail's input): a BR x 256 output tile holds whole
// rows of the tail's input. BR = 256 for large batches (the tiles of the
// separate layer), 64 for batches of fewer than one 256-row tile per CU.
// The layer is the 256 x 256 K loop of dense_relu_buf_kernel; its output
// (bias and ReLU in fp32) becomes hi/lo pairs in the LDS ring, which is free
// after the K loop (PR-row passes: 128 rows of hi, then of lo, 512 bytes a
// row, 16-byte chunk c of row r at slot c ^ (r & 7), so the tail's fragment
// reads of 8 rows hit 8 different slots), and the tail's two layers and head
// run on each pass, 8 waves each taking two 16-feature blocks of the first
// layer and one of the second over half of the pass's rows. A 256-row tile
// takes two passes: pass p holds row blocks 4p .. 4p + 3 of every wave's
// 128 rows, so each wave frees half of its accumulators per pass. The
// layer's output never goes to HBM.
template <typename TS, int BR, int MINB, int WN = 4, int KB = 64, int S = 2>
__global__ __launch_bounds__(128 * WN, MINB) void dense_tail_kernel(
    const TS *__restrict__ X, const TS *__restrict__ W, const float *__restrict__ bias, int64_t R,
    int K, int tiles_total, const TS *__restrict__ W1, const float *__restrict__ b1,
    const TS *__restrict__ W2, const float *__restrict__ b2, const TS *__restrict__ Wh,
    const float *__restrict__ bh, int n_out, float *__restrict__ scores) {
  typedef typename Mfma<TS>::frag frag;
  constexpr int BN = 256;
  typedef BufTile<BR, BN, S, WN, KB> G;
  constexpr int NI = G::NI, RJ = G::RJ, NT = G::NT;
  constexpr int N1 = 128, N2 = 64;                     // tail widths
  constexpr int S1 = N1 + 8, S2 = N2 + 4;              // padded LDS rows of the tail
  constexpr int HROW = BN * 2;                         // bytes per row of the layer's output
  constexpr int KS1 = BN / 32, KS2 = N1 / 32;
  // rows per pass: as many as the ring holds as hi/lo pairs, at most 128
  constexpr int PR = BR <= 128 && 2 * BR * HROW <= G::RING ? BR : (2 * 128 * HROW <= G::RING ? 128 : 64);
  constexpr int NP = BR / PR, JP = RJ / NP;            // passes; row blocks of a wave per pass
  constexpr int RH = G::NW / 4;                        // row groups of the tail layers
  constexpr int JB = PR / RH / 16;                     // row blocks of a wave in the tail layers
  constexpr int H3_BYTES = 2 * PR * HROW;              // hi and lo of the layer's output
  constexpr int H1_BYTES = 2 * PR * S1 * 2, H2_BYTES = PR * S2 * 4;
  // head weights in the ring when it has room past the layer's output
  constexpr bool WH_IN_RING = G::RING >= H3_BYTES + 2 * N2 * 4 + 16;
  static_assert(G::RING >= H3_BYTES, "a pass of the layer's output takes the ring");
  static_assert(G::NW == 4 || G::NW == 8, "the tail layers split 4 (features) x NW / 4 (rows)");
  static_assert(H1_BYTES + H2_BYTES <= H3_BYTES, "both hidden tiles fit where the layer's output was");
  static_assert(RJ % NP == 0 && PR * 4 <= NT && JB >= 1, "passes");
  __shared__ __align__(16) unsigned char smem[G::RING];
  __shared__ float s_whb_own[WH_IN_RING ? 1 : 2 * N2 + 4];
  float *s_wh = WH_IN_RING ? reinterpret_cast<float *>(smem + H3_BYTES) : s_whb_own;
  float *s_bh = s_wh + 2 * N2;

  const int tile = xcd_tile(blockIdx.x, tiles_total);
  const int64_t r0 = (int64_t)tile * BR;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave % WN, wr = wave / WN;

  // tail weights: wave w owns feature blocks 2 (w % 4) and 2 (w % 4) + 1 of
  // the first tail layer, and feature block w % 4 of the second, each on
  // the rows PR/2 (w / 4) .. PR/2 (w / 4 + 1) of a pass. With few
  // accumulators they are loaded before the K loop, so their latency hides
  // behind it (the loads are older than the ring's, which the K loop's
  // counted waits allow for); with many, after it.
  constexpr bool W_EARLY = NI * RJ <= 8;
  frag w1f[KS1][2], w2f[KS2][1];
  float whv, bhv;
  auto load_tail_weights = [&]() {
#pragma unroll
    for (int k = 0; k < KS1; ++k)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        w1f[k][i] = *reinterpret_cast<const frag *>(W1 + frag_offset(2 * (wave % 4) + i, k, KS1, lane));
#pragma unroll
    for (int k = 0; k < KS2; ++k)
      w2f[k][0] = *reinterpret_cast<const frag *>(W2 + frag_offset(wave % 4, k, KS2, lane));
    whv = Elem<TS>::to_f32(Wh[tid < n_out * N2 ? tid : 0]);
    bhv = bh[tid < n_out ? tid : 0];
  };
  if constexpr (W_EARLY) load_tail_weights();

  f32x4 acc[NI][RJ];
  buf_tile_kloop<TS, BR, BN, S, WN, KB>(X, W, bias, R, BN, K, r0, 0, smem, acc);
  if constexpr (!W_EARLY) load_tail_weights();
  compiler_fence();
  __builtin_amdgcn_s_barrier();   // every wave is past the K loop: the ring is free
  compiler_fence();
  if (tid < n_out * N2) s_wh[tid] = whv;
  if (tid < n_out) s_bh[tid] = bhv;

  const int dn = (lane >> 4) * 4, dr = lane & 15;
  TS *s_h1 = reinterpret_cast<TS *>(smem);
  float *s_h2 = reinterpret_cast<float *>(smem + H1_BYTES);
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    // this pass's rows of the layer's output: bias (in the accumulators),
    // ReLU, hi/lo pairs into the LDS
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int n = wn * (BN / WN) + i * 16 + dn;
#pragma unroll
      for (int jj = 0; jj < JP; ++jj) {
        const int j = p * JP + jj;
        const int rl = wr * (PR / 2) + jj * 16 + dr;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][e] > 0.0f ? acc[i][j][e] : 0.0f;
        uint2 hi, lo;
        split2<TS>(v[0], v[1], hi.x, lo.x);
        split2<TS>(v[2], v[3], hi.y, lo.y);
        unsigned char *o = smem + rl * HROW + (((n >> 3) ^ (rl & 7)) << 4) + (n & 7) * 2;
        *reinterpret_cast<uint2 *>(o) = hi;
        *reinterpret_cast<uint2 *>(o + PR * HROW) = lo;
      }
    }
    __syncthreads();   // the pass's tile (and the head weights) are in the LDS

    // first tail layer (each wave reads its row group of the pass once for
    // its two feature blocks); the tile is dead once every wave has its
    // sums, and the layer's output takes its place
    auto in0 = [&](int row, int c) {
      return reinterpret_cast<const TS *>(smem + row * HROW + ((c ^ (row & 7)) << 4));
    };
    f32x4 a1[2][JB];
    tail_mma<TS, KS1, 2, JB, true>(in0, PR * HROW, w1f, (wave / 4) * JB, lane, a1);
    __syncthreads();
    tail_store_ext<TS, 2, JB>(a1, b1, s_h1, S1, PR * S1, 2 * (wave % 4), (wave / 4) * JB, lane);
    __syncthreads();
    // second tail layer (wave w: feature block fb = w % 4 over its row
    // group), bias and ReLU in fp32, and the head's sums over the block's 16
    // features straight from the accumulators: lane (c, q) holds features
    // 16 fb + 4 q + e of row c; its four products are added in e order, the
    // four quarters by two shuffles; the feature blocks' sums meet in LDS
    auto in1 = [&](int row, int c) { return s_h1 + row * S1 + c * 8; };
    f32x4 a2[1][JB];
    tail_mma<TS, KS2, 1, JB, true>(in1, PR * S1 * 2, w2f, (wave / 4) * JB, lane, a2);
    {
      const int fb = wave % 4, q4 = lane >> 4;
      float wz0[4], wz1[4], bb[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int k = 16 * fb + 4 * q4 + e;
        wz0[e] = s_wh[k];
        wz1[e] = n_out > 1 ? s_wh[N2 + k] : 0.0f;
        bb[e] = b2[k];
      }
#pragma unroll
      for (int j = 0; j < JB; ++j) {
        float z0 = 0.0f, z1 = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = a2[0][j][e] + bb[e];
          v = v > 0.0f ? v : 0.0f;
          z0 += wz0[e] * v;
          z1 += wz1[e] * v;
        }
        z0 += __shfl_xor(z0, 16);
        z0 += __shfl_xor(z0, 32);
        z1 += __shfl_xor(z1, 16);
        z1 += __shfl_xor(z1, 32);
        if (q4 == 0) {
          const int lr = ((wave / 4) * JB + j) * 16 + dr;
          s_h2[(fb * PR + lr) * 2] = z0;
          s_h2[(fb * PR + lr) * 2 + 1] = z1;
        }
      }
    }
    __syncthreads();
    // head: the four blocks' sums in block order, then the bias; LDS row lr
    // of the pass is row (lr / (PR/2)) * (BR/2) + p * (PR/2) + lr % (PR/2) of
    // the tile
    if (tid < PR) {
      const int lr = tid;
      float z0 = s_h2[lr * 2], z1 = s_h2[lr * 2 + 1];
#pragma unroll
      for (int fb = 1; fb < 4; ++fb) {
        z0 += s_h2[(fb * PR + lr) * 2];
        z1 += s_h2[(fb * PR + lr) * 2 + 1];
      }
      const int64_t r = r0 + (lr / (PR / 2)) * (BR / 2) + p * (PR / 2) + lr % (PR / 2);
      if (r < R) {
        z0 += s_bh[0];
        if (n_out > 1) z1 += s_bh[1];
        scores[r] = n_out == 1 ? 1.0f / (1.0f + expf(-z0)) : 1.0f / (1.0f + expf(z0 - z1));
      }
    }
    if (p + 1 < NP) __syncthreads();   // the next pass overwrites the tail's tiles
  }
}

// fp32 layer: 64 x 64 output tile, 4 x 4 per thread, K in chunks of 128
// staged in LDS; each thread loads its part of the next chunk into
// registers before it computes on the current one, so a layer of K <= 128
// costs one memory round trip, not one per 16-deep step. Sums over k in
// index order.
constexpr int kF32Chunk = 128;
__global__ __launch_bounds__(256) void dense_relu_f32_kernel(const float *__restrict__ X,
                                                             const float *__restrict__ W,
                                                             const float *__restrict__ bias,
                                                             float *__restrict__ Y, int64_t R,
                                                             int N, int K, int relu) {
  constexpr int KC = kF32Chunk, PER = 64 * KC / 256;   // elements of each operand per thread
  __shared__ float sx[KC][64 + 1];
  __shared__ float sw[KC][64 + 1];
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  const int n0 = blockIdx.y * 64;
  const int tr = tid >> 4, tn = tid & 15;
  float acc[4][4] = {};
  float vx[PER], vw[PER];
  auto load = [&](int k0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + u * 256;
      const int row = i / KC, kk = i % KC;
      const int64_t r = r0 + row;
      const int n = n0 + row, k = k0 + kk;
      vx[u] = (r < R && k < K) ? X[r * K + k] : 0.0f;
      vw[u] = (n < N && k < K) ? W[(int64_t)n * K + k] : 0.0f;
    }
  };
  load(0);
  for (int k0 = 0; k0 < K; k0 += KC) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int i = tid + u * 256;
      const int row = i / KC, kk = i % KC;
      sx[kk][row] = vx[u];
      sw[kk][row] = vw[u];
    }
    __syncthreads();
    if (k0 + KC < K) load(k0 + KC);
    const int kn = K - k0 < KC ? K - k0 : KC;
    for (int kk = 0; kk < kn; ++kk) {
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

// Y = act(X W^T + b) in fp32 on the matrix cores (v_mfma_f32_16x16x4_f32),
// without LDS: each wave owns 16 rows x 16*NB outputs and loads its operands
// straight into registers as 16-byte vectors.  In a 16-deep K chunk, lane l
// (row or output l % 16, quarter q = l / 16) holds k = 16c + 4q .. 4q + 3 of
// both operands, and the four MFMAs of the chunk take component 0, 1, 2, 3:
// every k of the chunk meets its partner exactly once (the order of the sum
// over k is permuted, which only moves fp32 rounding).  Four chunks are
// loaded before their MFMAs so one memory latency covers 64 of K.  act 0:
// none, 1: ReLU, 2: sigmoid.  Used for the SE layer of the literal Eq. 2
// form (one FC from the concatenated embedding to the M weights).  K must
// be a multiple of 4 (16-byte rows).
template <int ACT, int NB>
__global__ __launch_bounds__(256) void dense_f32_mfma_kernel(const float *__restrict__ X,
                                                             const float *__restrict__ W,
                                                             const float *__restrict__ bias,
                                                             float *__restrict__ Y, int64_t R, int N,
                                                             int K) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t rbase = (int64_t)blockIdx.x * 64 + wave * 16;
  const int nbase = blockIdx.y * (16 * NB);
  const int fr = lane & 15, q = lane >> 4;
  int64_t xr = rbase + fr;
  xr = xr < R ? xr : R - 1;                   // clamped: loaded, never stored
  const float *xp = X + xr * K + 4 * q;
  const float *wp[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    int n = nbase + i * 16 + fr;
    n = n < N ? n : N - 1;
    wp[i] = W + (int64_t)n * K + 4 * q;
  }
  f32x4 acc[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto ld = [&](const float *p, int k) -> float4 {   // k: chunk start; zero past K
    return (k + 4 * q < K) ? *reinterpret_cast<const float4 *>(p + k) : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  for (int k0 = 0; k0 < K; k0 += 64) {
    float4 xv[4], wv[4][NB];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      xv[c] = ld(xp, k0 + 16 * c);
#pragma unroll
      for (int i = 0; i < NB; ++i) wv[c][i] = ld(wp[i], k0 + 16 * c);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float xs[4] = {xv[c].x, xv[c].y, xv[c].z, xv[c].w};
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const float ws[4] = {wv[c][i].x, wv[c][i].y, wv[c][i].z, wv[c][i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(ws[e], xs[e], acc[i], 0, 0, 0);
      }
    }
  }
  // lane holds D[4 (lane/16) + e][lane % 16]: output feature, then row
  const int64_t r = rbase + fr;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = nbase + i * 16 + 4 * q + e;
      if (r < R && n < N) {
        float t = acc[i][e] + bias[n];
        if (ACT == 1) t = t > 0.0f ? t : 0.0f;
        if (ACT == 2) t = 1.0f / (1.0f + expf(-t));
        Y[r * N + n] = t;
      }
    }
}

template <int ACT>
static hipError_t launch_dense_f32_act(const float *x, const float *w, const float *b, float *y,
                                       int64_t R, int32_t N, int32_t K, hipStream_t s) {
  const unsigned gx = (unsigned)((R + 63) / 64);
  // fewer 64-row blocks than CUs: one 16-wide output block per wave and the
  // output blocks over the grid's second dimension, for more workgroups
  // (the sum over k runs in the same order whatever a wave's blocks)
  const int cus = device_cus() > 0 ? device_cus() : 256;
  if ((int64_t)gx < cus && N > 16) {
    hipLaunchKernelGGL((dense_f32_mfma_kernel<ACT, 1>), dim3(gx, (unsigned)((N + 15) / 16)), dim3(256), 0, s,
                       x, w, b, y, R, N, K);
    return hipGetLastError();
  }
  if (N <= 16) hipLaunchKernelGGL((dense_f32_mfma_kernel<ACT, 1>), dim3(gx, 1), dim3(256), 0, s, x, w, b, y, R, N, K);
  else if (N <= 32) hipLaunchKernelGGL((dense_f32_mfma_kernel<ACT, 2>), dim3(gx, 1), dim3(256), 0, s, x, w, b, y, R, N, K);
  else if (N <= 48) hipLaunchKernelGGL((dense_f32_mfma_kernel<ACT, 3>), dim3(gx, 1), dim3(256), 0, s, x, w, b, y, R, N, K);
  else hipLaunchKernelGGL((dense_f32_mfma_kernel<ACT, 4>), dim3(gx, (unsigned)((N + 63) / 64)), dim3(256), 0, s, x, w, b, y, R, N, K);
  return hipGetLastError();
}

hipError_t launch_dense_f32(const float *x, const float *w, const float *b, float *y, int64_t R,
                            int32_t N, int32_t K, int act, hipStream_t s) {
  if (R <= 0 || N <= 0) return hipSuccess;
  if (K % 4 != 0) return hipErrorInvalidValue;
  if (act == 2) return launch_dense_f32_act<2>(x, w, b, y, R, N, K, s);
  if (act == 1) return launch_dense_f32_act<1>(x, w, b, y, R, N, K, s);
  return launch_dense_f32_act<0>(x, w, b, y, R, N, K, s);
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
template <typename TS, int BR, int BN>
static hipError_t dense_mfma_t(const void *x, const void *w, const float *b, void *y, int64_t R,
                               int N, int K, hipStream_t s) {
  const int tiles_n = (N + BN - 1) / BN;
  const int64_t tiles_r = (R + BR - 1) / BR;
  const int64_t total = tiles_r * tiles_n;
  if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dense_relu_mfma_kernel<TS, BR, BN>), dim3((unsigned)total), dim3(256), 0, s,
                     static_cast<const TS *>(x), static_cast<const TS *>(w), b,
                     static_cast<TS *>(y), R, N, K, tiles_n, (int)total);
  return hipGetLastError();
}

// requests with weights of their own (see dense_relu_buf_kernel's GRP)
struct GroupArgs {
  int64_t Q;
  RowTile *tiles;
  int32_t *n_tiles;
  int64_t w_stride;
};

template <typename TS, int BR, int BN, int S, int WN, int MINW, int KB, bool HALF>
static hipError_t dense_buf_launch(const void *x, const void *w, const float *b, void *y, int64_t R,
                                   int N, int K, hipStream_t s, const GroupArgs *ga) {
  const int tiles_n = (N + BN - 1) / BN;
  const int64_t tiles_r = ga ? row_tiles_bound(R, ga->Q, BR) : (R + BR - 1) / BR;
  const int64_t total = tiles_r * tiles_n;
  if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
  if (ga) {
    hipLaunchKernelGGL((dense_relu_buf_kernel<TS, BR, BN, S, WN, MINW, KB, true, HALF>), dim3((unsigned)total),
                       dim3(128 * WN), 0, s, static_cast<const TS *>(x), static_cast<const TS *>(w), b,
                       static_cast<TS *>(y), R, N, K, tiles_n, (int)total, ga->tiles, ga->n_tiles,
                       ga->w_stride);
  } else {
    hipLaunchKernelGGL((dense_relu_buf_kernel<TS, BR, BN, S, WN, MINW, KB, false, HALF>), dim3((unsigned)total),
                       dim3(128 * WN), 0, s, static_cast<const TS *>(x), static_cast<const TS *>(w), b,
                       static_cast<TS *>(y), R, N, K, tiles_n, (int)total,
                       static_cast<const RowTile *>(nullptr), static_cast<const int32_t *>(nullptr),
                       (int64_t)0);
  }
  return hipGetLastError();
}

// 64-deep stages take the half-stage variant when K % 64 == 32
template <typename TS, int BR, int BN, int S, int WN, int MINW, int KB = 32>
static hipError_t dense_buf_t(const void *x, const void *w, const float *b, void *y, int64_t R,
                              int N, int K, hipStream_t s, const GroupArgs *ga = nullptr) {
  if constexpr (KB == 64) {
    if (K % 64 != 0) return dense_buf_launch<TS, BR, BN, S, WN, MINW, 64, true>(x, w, b, y, R, N, K, s, ga);
  }
  return dense_buf_launch<TS, BR, BN, S, WN, MINW, KB, false>(x, w, b, y, R, N, K, s, ga);
}

// The tile shape of a layer of R rows, N outputs and K inputs (the
// buffered kernel for K % 32 == 0 and N % 8 == 0, else the plain one).
//   Large batches: 256 x 256 tiles over 8 waves, in 64-deep stages (one
// barrier per 64 MFMAs per wave, whole 128-byte rows per load; a last half
// stage when K % 64 == 32), or 256 x 128 and 256 x 64 over 4 waves in
// 32-deep stages for narrower layers; batches of a few thousand ads would
// leave most CUs idle with those, so 128..192 x 128 tiles while 128-row
// tiles would still number one per CU, else 64 x 64.
//   Every tile shape sums the same 32-deep K blocks in the same order, so the
// outputs do not depend on the shape.
enum class DTile {
  k192x128, k160x128, k128x128, k64x64_3s, k64x64, k256x256, k256x128, k256x64, kPlain128, kPlain64
};

static DTile dense_tile(int64_t R, int N, int K) {
  if (K % kBK != 0 || N % 8 != 0) return N % 128 == 0 ? DTile::kPlain128 : DTile::kPlain64;
  const int64_t big_tiles = ((R + 255) / 256) * ((N + 127) / 128);
  const int64_t mid_tiles = ((R + 127) / 128) * ((N + 127) / 128);
  // 64-deep stages for every K here (K % 32 == 0; a half stage ends K % 64 == 32)
  const int64_t cus = device_cus() > 0 ? device_cus() : 256;
  if (big_tiles < 256 && mid_tiles >= 256 && N % 128 == 0) {
    // x 128 tiles with the row height that gives the least work to the
    // busiest CU (rounds of one tile per CU), provided the tiles still
    // cover three quarters of the CUs (fewer, smaller layers run faster on
    // 64 x 64 tiles, two per CU)
    const int heights[3] = {192, 160, 128};
    int best = 0;
    int64_t best_cost = -1;
    for (int h : heights) {
      const int64_t tiles = ((R + h - 1) / h) * (N / 128);
      const int64_t cost = (tiles + cus - 1) / cus * h;
      if (4 * tiles >= 3 * cus && (best_cost < 0 || cost < best_cost)) best = h, best_cost = cost;
    }
    if (best == 192) return DTile::k192x128;
    if (best == 160) return DTile::k160x128;
    return DTile::k128x128;
  }
  if (big_tiles < 256) {
    // at most two tiles per CU: a third 64-deep stage in flight (the K steps
    // wait on load latency, not on the CU's throughput); more tiles than
    // that run better with the smaller ring, more workgroups per CU
    const int64_t small_tiles = ((R + 63) / 64) * ((N + 63) / 64);
    return small_tiles <= 2 * cus ? DTile::k64x64_3s : DTile::k64x64;
  }
  if (N % 256 == 0) return DTile::k256x256;
  return N % 128 == 0 ? DTile::k256x128 : DTile::k256x64;
}

// rows of a tile (the buffered shapes)
static int dense_tile_rows(DTile t) {
  switch (t) {
    case DTile::k192x128: return 192;
    case DTile::k160x128: return 160;
    case DTile::k128x128: return 128;
    case DTile::k64x64_3s: case DTile::k64x64: return 64;
    default: return 256;
  }
}

template <typename TS>
static hipError_t dense_mfma_dt(const void *x, const void *w, const float *b, void *y, int64_t R,
                                int N, int K, hipStream_t s, const GroupArgs *ga = nullptr) {
  switch (dense_tile(R, N, K)) {
    case DTile::k192x128: return dense_buf_t<TS, 192, 128, 2, 2, 2, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k160x128: return dense_buf_t<TS, 160, 128, 2, 2, 2, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k128x128: return dense_buf_t<TS, 128, 128, 2, 2, 2, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k64x64_3s: return dense_buf_t<TS, 64, 64, 3, 2, 2, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k64x64: return dense_buf_t<TS, 64, 64, 2, 2, 2, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k256x256: return dense_buf_t<TS, 256, 256, 2, 4, 1, 64>(x, w, b, y, R, N, K, s, ga);
    case DTile::k256x128: return dense_buf_t<TS, 256, 128, 3, 2, 2>(x, w, b, y, R, N, K, s, ga);
    case DTile::k256x64: return dense_buf_t<TS, 256, 64, 3, 2, 2>(x, w, b, y, R, N, K, s, ga);
    case DTile::kPlain128:
      if (ga) return hipErrorInvalidValue;
      return dense_mfma_t<TS, 256, 128>(x, w, b, y, R, N, K, s);
    default:
      if (ga) return hipErrorInvalidValue;
      return dense_mfma_t<TS, 256, 64>(x, w, b, y, R, N, K, s);
  }
}

hipError_t launch_dense_relu(int dtype, const void *x, const void *w, const float *b, void *y,
                             int64_t R, int32_t N, int32_t K, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (dtype == kF32) {
    // fp32 models: the fp32 matrix cores when rows are whole 16-byte vectors
    if (K % 4 == 0)
      return launch_dense_f32(static_cast<const float *>(x), static_cast<const float *>(w), b,
                              static_cast<float *>(y), R, N, K, 1, s);
    const dim3 grid((unsigned)((R + 63) / 64), (unsigned)((N + 63) / 64));
    hipLaunchKernelGGL(dense_relu_f32_kernel, grid, dim3(256), 0, s, static_cast<const float *>(x),
                       static_cast<const float *>(w), b, static_cast<float *>(y), R, N, K, 1);
    return hipGetLastError();
  }
  if (dtype == kBF16) return dense_mfma_dt<__bf16>(x, w, b, y, R, N, K, s);
  return dense_mfma_dt<_Float16>(x, w, b, y, R, N, K, s);
}

bool dense_grouped_supported(int dtype, int32_t N, int32_t K) {
  return dtype != kF32 && K > 0 && K % kBK == 0 && N > 0 && N % 8 == 0;
}

hipError_t launch_dense_relu_grouped(int dtype, const void *x, const void *w, const float *b,
                                     void *y, int64_t R, int64_t Q, int32_t N, int32_t K,
                                     RowTile *tiles, int32_t *n_tiles, hipStream_t s) {
  if (R <= 0 || Q <= 0) return hipSuccess;
  if (!dense_grouped_supported(dtype, N, K)) return hipErrorInvalidValue;
  const GroupArgs ga{Q, tiles, n_tiles, (int64_t)N * K};
  if (dtype == kBF16) return dense_mfma_dt<__bf16>(x, w, b, y, R, N, K, s, &ga);
  return dense_mfma_dt<_Float16>(x, w, b, y, R, N, K, s, &ga);
}

int dense_grouped_tile_rows(int64_t R, int32_t N, int32_t K) {
  return dense_tile_rows(dense_tile(R, N, K));
}

bool tail_supported(int dtype, int K0, int N1, int N2, int n_out) {
  return dtype != kF32 && K0 == 256 && N1 == 128 && N2 == 64 && (n_out == 1 || n_out == 2);
}

template <typename TS>
static void launch_tail_t(const void *a, const void *w1, const float *b1, const void *w2,
                          const float *b2, const void *wh, const float *bh, int32_t n_out,
                          float *scores, int64_t R, hipStream_t s) {
  hipLaunchKernelGGL((mlp_tail_kernel<TS, 256, 128, 64>), dim3((unsigned)((R + 63) / 64)),
                     dim3(256), 0, s, static_cast<const TS *>(a), static_cast<const TS *>(w1), b1,
                     static_cast<const TS *>(w2), b2, static_cast<const TS *>(wh), bh, n_out,
                     scores, R);
}

hipError_t launch_mlp_tail(int dtype, const void *a, const void *w1, const float *b1,
                           const void *w2, const float *b2, const void *wh, const float *bh,
                           int32_t n_out, float *scores, int64_t R, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (dtype == kBF16) launch_tail_t<__bf16>(a, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
  else launch_tail_t<_Float16>(a, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
  return hipGetLastError();
}

bool dense_tail_supported(int dtype, int64_t R, int32_t N, int32_t K) {
  // the layer's output is the tail's 256-wide input, in 64-deep K steps
  return dtype != kF32 && N == 256 && K > 0 && K % 64 == 0 && R > 0 && (R + 63) / 64 <= 0x7FFFFFFF;
}

template <typename TS, int BR, int MINB, int WN = 4, int KB = 64, int S = 2>
static void launch_dense_tail_t(const void *x, const void *w, const float *b, int32_t K,
                                const void *w1, const float *b1, const void *w2, const float *b2,
                                const void *wh, const float *bh, int32_t n_out, float *scores,
                                int64_t R, hipStream_t s) {
  const int tiles = (int)((R + BR - 1) / BR);
  hipLaunchKernelGGL((dense_tail_kernel<TS, BR, MINB, WN, KB, S>), dim3(tiles), dim3(128 * WN), 0, s,
                     static_cast<const TS *>(x), static_cast<const TS *>(w), b, R, K, tiles,
                     static_cast<const TS *>(w1), b1, static_cast<const TS *>(w2), b2,
                     static_cast<const TS *>(wh), bh, n_out, scores);
}

hipError_t launch_dense_tail(int dtype, const void *x, const void *w, const float *b, int32_t N,
                             int32_t K, const void *w1, const float *b1, const void *w2,
                             const float *b2, const void *wh, const float *bh, int32_t n_out,
                             float *scores, int64_t R, hipStream_t s) {
  if (!dense_tail_supported(dtype, R, N, K)) return hipErrorNotSupported;
  // 256-row tiles over 8 waves while the separate layer would use 256 x 256
  // tiles (at least one tile per CU); for batches of many rounds of tiles,
  // 128-row tiles over 4 waves in 72 KB of LDS, two workgroups per CU, so
  // that one's tail phase overlaps the other's K loop (the large workload,
  // 1.28 M rows: 720 -> 650 us; at 64,000 rows, one round, 40 -> 42 us);
  // 64-row tiles for smaller batches, and 32-row tiles over 4 waves when
  // 64-row tiles would leave CUs idle. Every variant sums in the same order.
  const bool big = ((R + 255) / 256) * 2 >= 256;
  const int cus = device_cus() > 0 ? device_cus() : 256;
  const bool rounds = (R + 127) / 128 >= 8 * (int64_t)cus;
  const bool few = (R + 63) / 64 < cus;
  if (dtype == kBF16) {
    if (big && rounds) launch_dense_tail_t<__bf16, 128, 2, 2, 32, 3>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else if (big) launch_dense_tail_t<__bf16, 256, 1>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else if (few) launch_dense_tail_t<__bf16, 32, 2, 2>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else launch_dense_tail_t<__bf16, 64, 2>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
  } else {
    if (big && rounds) launch_dense_tail_t<_Float16, 128, 2, 2, 32, 3>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else if (big) launch_dense_tail_t<_Float16, 256, 1>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else if (few) launch_dense_tail_t<_Float16, 32, 2, 2>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
    else launch_dense_tail_t<_Float16, 64, 2>(x, w, b, K, w1, b1, w2, b2, wh, bh, n_out, scores, R, s);
  }
  return hipGetLastError();
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
