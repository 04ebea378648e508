// gfx950 kernels of the greedy speculative-verification step.
//
// One verify step runs the target model over a block of T <= 513 rows (the
// pending token plus up to 512 draft tokens, Eq. 3), decodes every row
// greedily and accepts the longest matching draft prefix (Eq. 7).  Weight
// streaming dominates: every linear layer is a skinny GEMM with T rows, so
// each weight byte is read once per step and the GEMMs are HBM-bound.
//
// Arithmetic layout (identical for every T, so a row's result never depends
// on how many other rows share its block; a K = 0 step and a K = 64 step give
// bitwise-equal rows):
//   * GEMM: weights are the MFMA A operand (16 output features per tile),
//     activations the B operand (16 rows per t-tile).  A workgroup's 8 waves
//     take the super-steps of its part of the reduction round-robin and are
//     summed in wave order; K slices (down projection, LM head, d > 4096) are
//     added in slice order by the consuming kernel.
//   * Attention: keys in splits of 256 absolute positions, each split in
//     64-position sub-tiles combined by an online softmax in order; splits
//     merged in order by a second kernel.
//   * Residual stream, accumulators, softmax and logits are fp32; bf16 models
//     round the projections' inputs h * gain, q/k after rotary, v, the
//     attention output and the SwiGLU product to bf16 (nearest-even).

#include "kernels.h"

#include <hip/hip_runtime.h>
#include <math.h>

#include <algorithm>

namespace ee {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));


// ---------------------------------------------------------------- numerics --

__device__ __forceinline__ uint32_t f2bf_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;   // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                        // nearest, ties to even
  return u >> 16;
}
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }
// Sum and maximum of x over the lanes l, l ^ 16 (row pairs) or l, l ^ 32
// (halves) of a wave with v_permlane16_swap / v_permlane32_swap: the swap
// leaves x[l] and x[l ^ 16] (x[l ^ 32]) in its two results of every lane, in
// the same order for both lanes of a pair, so the value is that of
// x + shfl_xor(x, 16) (32) without the LDS round trip.
__device__ __forceinline__ float xsum16(float x) {
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
__device__ __forceinline__ float xsum32(float x) {
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
__device__ __forceinline__ float xmax16(float x) {
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
__device__ __forceinline__ float xmax32(float x) {
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
// Nearest-even bf16 bits of two finite floats, a in the low half, with one
// v_cvt_pk_bf16_f32 (equal to f2bf_bits_finite of each, checked for every
// finite float bit pattern).
__device__ __forceinline__ uint32_t bf16x2_bits(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}
// Nearest-even bf16 bits of a finite float (no NaN handling, no branch).
__device__ __forceinline__ uint32_t f2bf_bits_finite(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Round a float to the storage type and return the stored value as float.
template <int DT> __device__ __forceinline__ float rnd(float x);
template <> __device__ __forceinline__ float rnd<DT_F32>(float x) { return x; }
template <> __device__ __forceinline__ float rnd<DT_BF16>(float x) { return bf2f(f2bf_bits(x)); }

template <int DT> __device__ __forceinline__ void store_elt(void* base, size_t i, float x);
template <> __device__ __forceinline__ void store_elt<DT_F32>(void* base, size_t i, float x) {
  reinterpret_cast<float*>(base)[i] = x;
}
template <> __device__ __forceinline__ void store_elt<DT_BF16>(void* base, size_t i, float x) {
  reinterpret_cast<uint16_t*>(base)[i] = (uint16_t)f2bf_bits(x);
}
template <int DT> __device__ __forceinline__ float load_elt(const void* base, size_t i);
template <> __device__ __forceinline__ float load_elt<DT_F32>(const void* base, size_t i) {
  return reinterpret_cast<const float*>(base)[i];
}
template <> __device__ __forceinline__ float load_elt<DT_BF16>(const void* base, size_t i) {
  return bf2f(reinterpret_cast<const uint16_t*>(base)[i]);
}

template <int DT> struct Geo;
template <> struct Geo<DT_BF16> { static constexpr int KS = 32, EPL = 8, ESZ = 2; };
template <> struct Geo<DT_F32> { static constexpr int KS = 16, EPL = 4, ESZ = 4; };

// D += A * B over one fragment pair (16x16 tile, KS reduction columns).
template <int DT> __device__ __forceinline__ f32x4 mma(uint4 a, uint4 b, f32x4 c);
template <> __device__ __forceinline__ f32x4 mma<DT_BF16>(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ __forceinline__ f32x4 mma<DT_F32>(uint4 a, uint4 b, f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

// Element index, inside a packed fragment buffer with S super-steps, of
// matrix element (row, col).
template <int DT> __device__ __forceinline__ size_t frag_index(int row, int col, int S) {
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL;
  const int tt = row >> 4, c = row & 15;
  const int s = col / KS, kk = col % KS;
  const int grp = kk / EPL, e = kk % EPL;
  return ((size_t)(tt * S + s) * 64 + grp * 16 + c) * EPL + e;
}

// ------------------------------------------------------------------ packing --

template <int DT>
__global__ void pack_kernel(const void* __restrict__ src, int rows, int dst_row0, int K,
                            uint4* __restrict__ dst) {
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL;
  const int S = K / KS;
  // one thread per destination lane-fragment (16 bytes)
  const size_t frags = (size_t)rows / 16 * S * 64;
  for (size_t f = blockIdx.x * (size_t)blockDim.x + threadIdx.x; f < frags;
       f += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(f & 63);
    const size_t ts = f >> 6;
    const int s = (int)(ts % S);
    const int tile_local = (int)(ts / S);
    const int grp = lane >> 4, c = lane & 15;
    const int sr = tile_local * 16 + c;
    const int col0 = s * KS + grp * EPL;   // EPL elements = 16 bytes, 16-byte aligned
    const uint4 v = *reinterpret_cast<const uint4*>(reinterpret_cast<const unsigned char*>(src) +
                                                    ((size_t)sr * K + col0) * Geo<DT>::ESZ);
    const size_t dtile = (size_t)(dst_row0 / 16 + tile_local);
    dst[(dtile * S + s) * 64 + lane] = v;
  }
}

hipError_t launch_pack(const PackSrc& ps, void* dst, int K, int dt, hipStream_t st) {
  const int ks = ks_of(dt);
  if (K % ks || ps.rows % 16 || ps.dst_row0 % 16) return hipErrorInvalidValue;
  const size_t frags = (size_t)ps.rows / 16 * (K / ks) * 64;
  const int threads = 256;
  const size_t want = (frags + threads - 1) / threads;
  const int blocks = (int)(want < 65536 ? want : 65536);
  if (dt == DT_BF16)
    hipLaunchKernelGGL(pack_kernel<DT_BF16>, dim3(blocks), dim3(threads), 0, st, ps.src, ps.rows,
                       ps.dst_row0, K, reinterpret_cast<uint4*>(dst));
  else
    hipLaunchKernelGGL(pack_kernel<DT_F32>, dim3(blocks), dim3(threads), 0, st, ps.src, ps.rows,
                       ps.dst_row0, K, reinterpret_cast<uint4*>(dst));
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
  return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st);
}

// -------------------------------------------------------------------- GEMM --
//
// Y[t, n] = sum_k X[t, k] W[n, k] for T <= 80 rows, split over K:
//   * the reduction dimension (S super-steps of KS columns) is cut into SK
//     slices of SS super-steps; SK depends only on (N, K);
//   * a workgroup (8 waves) owns one slice and a set of 16-feature tiles;
//     wave w accumulates the slice's super-steps w, w+8, w+16, ... in order,
//     holding its activation fragments in registers for the whole kernel and
//     streaming weight fragments one tile ahead;
//   * the 8 wave partials of a tile are summed in wave order and stored as
//     part[k][t][n]; the consumer kernel adds the SK slices in slice order.
// The arithmetic of an output element therefore never depends on T or on
// which workgroup computed it.

constexpr int GEMM_WAVES = 8;
constexpr int GEMM_SPW = 8;           // super-steps per wave per slice (max)
constexpr unsigned OOB = 0x80000000u; // buffer offset past every range: loads 0

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// 16-byte buffer load; offsets beyond the resource size return zeros without
// a memory access.  AUX selects the cache policy (2 = non-temporal).
template <int AUX>
__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, unsigned off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// 8-byte buffer load (as bload).
template <int AUX>
__device__ __forceinline__ uint2 bload64(__amdgpu_buffer_rsrc_t r, unsigned off) {
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX);
  return make_uint2(v.x, v.y);
}

struct GemmArgs {
  const uint4* w;       // packed weights [n_tiles][S][64]
  const uint4* x;       // packed activations of all Ttot rows [ceil(Ttot/16)][S][64]
  float* part;          // [SK][Ttot][N]
  int S, SK, SS, N, n_tiles;
  int Ttot;             // rows of the block
  int rows;             // rows per row group (a multiple of 16, at most 16 MT)
  int P, G;             // workgroups per row group (G tile groups x SK slices used), tile groups
};

inline int gemm_slices(int S) {
  int sk = 1;
  while (S > GEMM_SPW * GEMM_WAVES * sk) sk *= 2;
  return sk;   // <= 16 for every K the library accepts (K <= 32768)
}

// Workgroup (row group rg, tile group g, slice k) = blockIdx rg * P + g * SK + k
// holds the activation fragments of its rows for slice k in registers and
// streams the weight tiles g, g + G, ...  Every row group repeats the same
// weight stream; with P a multiple of 8 the workgroups that share a stream
// sit on the same XCD (workgroups are dealt to the 8 XCDs in turn) and run
// side by side, so one of them fetches each weight tile from HBM and the
// others find it in that XCD's L2.  NT: non-temporal weight loads (one row
// group: nothing re-reads them).
template <int DT, int MT, bool NT>
__global__ __launch_bounds__(GEMM_WAVES * 64) void gemm_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, c = lane & 15;
  const int rg = blockIdx.x / a.P, q = blockIdx.x - rg * a.P;
  if (q >= a.SK * a.G) return;
  const int k = q % a.SK, groups = a.G;
  const int row0 = rg * a.rows, T = min(a.rows, a.Ttot - row0);
  const int S = a.S, s0 = k * a.SS, ns = min(S - s0, a.SS);
  const auto xs = make_rsrc(a.x + (size_t)(row0 / 16) * S * 64, (unsigned)(MT * S * 1024));
  const auto ws = make_rsrc(a.w, (unsigned)((size_t)a.n_tiles * S * 1024));
  const auto ps = make_rsrc(a.part, (unsigned)((size_t)a.SK * a.Ttot * a.N * 4));
  constexpr int WAUX = NT ? 2 : 0;
  uint4 xr[GEMM_SPW][MT];
#pragma unroll
  for (int i = 0; i < GEMM_SPW; ++i) {
    const int sl = wv + GEMM_WAVES * i;
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (MT > 1)   // (one tile: requested with the first weights below)
        xr[i][m] = bload<0>(xs, (sl < ns && m * 16 + c < T)
                                    ? (unsigned)(((m * S + s0 + sl) * 64 + lane) * 16) : OOB);
  }
  auto wload = [&](int tl, int i) {
    const int sl = wv + GEMM_WAVES * i;
    return bload<WAUX>(ws, (tl < a.n_tiles && sl < ns) ? (unsigned)(((tl * S + s0 + sl) * 64 + lane) * 16) : OOB);
  };
  __shared__ f32x4 red[2][GEMM_WAVES][MT][64];
  // this thread's reduction item: fragment rm, lane rl (threads past MT * 64
  // repeat an item and store nothing: the loop body has no branch, so the
  // compiler never has to wait for the weights in flight at the loop edge)
  const int qq = threadIdx.x % (MT * 64);
  const bool qown = threadIdx.x < MT * 64;
  const int rm = qq >> 6, rl = qq & 63, rt = rm * 16 + (rl & 15);
  auto tile_step = [&](const uint4 (&wf)[GEMM_SPW], int tile, int pb) {
    f32x4 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < GEMM_SPW; ++i)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] = mma<DT>(wf[i], xr[i][m], acc[m]);
#pragma unroll
    for (int m = 0; m < MT; ++m) red[pb][wv][m][lane] = acc[m];
    __syncthreads();
    f32x4 v = red[pb][0][rm][rl];
#pragma unroll
    for (int j = 1; j < GEMM_WAVES; ++j) v += red[pb][j][rm][rl];
    const unsigned off = (qown && rt < T)
        ? (unsigned)((((size_t)k * a.Ttot + row0 + rt) * a.N + tile * 16 + 4 * (rl >> 4)) * 4) : OOB;
    __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(v.x), __float_as_uint(v.y),
                                                 __float_as_uint(v.z), __float_as_uint(v.w)}, ps, off, 0, 0);
  };
  // two named weight buffers: the next tile's fragments are requested before
  // the current tile is computed, and no in-flight register is ever copied
  int tile = q / a.SK;
  uint4 wa[GEMM_SPW], wb[GEMM_SPW];
  if (MT == 1) {
    // one row tile: inputs and the first tile's weights requested super-step
    // by super-step, in the order the first MFMAs use them
#pragma unroll
    for (int i = 0; i < GEMM_SPW; ++i) {
      const int sl = wv + GEMM_WAVES * i;
      xr[i][0] = bload<0>(xs, (sl < ns && c < T) ? (unsigned)(((s0 + sl) * 64 + lane) * 16) : OOB);
      wa[i] = wload(tile, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < GEMM_SPW; ++i) wa[i] = wload(tile, i);
  }
  for (;;) {
#pragma unroll
    for (int i = 0; i < GEMM_SPW; ++i) wb[i] = wload(tile + groups, i);
    tile_step(wa, tile, 0);
    tile += groups;
    if (tile >= a.n_tiles) break;
#pragma unroll
    for (int i = 0; i < GEMM_SPW; ++i) wa[i] = wload(tile + groups, i);
    tile_step(wb, tile, 1);
    tile += groups;
    if (tile >= a.n_tiles) break;
  }
}

constexpr int GEMM_MAX_ROWS = 80;   // rows one workgroup holds in registers (MT <= 5)

// Y = X W^T for R rows.  Up to 80 rows: one row group, one workgroup per CU,
// each streaming its weight tiles once.  More rows: groups of 80 rows in
// the same launch, sharing each weight stream through L2.  A row's
// arithmetic is the same either way (and the same as in a launch of its own).
template <int DT>
static hipError_t gemm(const uint4* w, const uint4* x, int N, int K, int R, float* part,
                       hipStream_t st) {
  GemmArgs a;
  a.w = w; a.x = x; a.part = part; a.N = N; a.Ttot = R;
  a.S = K / Geo<DT>::KS;
  a.SK = gemm_slices(a.S);
  a.SS = (a.S + a.SK - 1) / a.SK;
  a.n_tiles = N / 16;
  const dim3 block(GEMM_WAVES * 64);
  if (R <= GEMM_MAX_ROWS) {
    a.rows = R;
    a.G = std::max(1, std::min(256 / a.SK, a.n_tiles));
    a.P = a.G * a.SK;
    const dim3 grid(a.P);
    switch ((R + 15) / 16) {
      case 1: hipLaunchKernelGGL((gemm_kernel<DT, 1, true>), grid, block, 0, st, a); break;
      case 2: hipLaunchKernelGGL((gemm_kernel<DT, 2, true>), grid, block, 0, st, a); break;
      case 3: hipLaunchKernelGGL((gemm_kernel<DT, 3, true>), grid, block, 0, st, a); break;
      case 4: hipLaunchKernelGGL((gemm_kernel<DT, 4, true>), grid, block, 0, st, a); break;
      case 5: hipLaunchKernelGGL((gemm_kernel<DT, 5, true>), grid, block, 0, st, a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  a.rows = GEMM_MAX_ROWS;
  const int rg = (R + GEMM_MAX_ROWS - 1) / GEMM_MAX_ROWS;
  a.P = std::max(256 / rg / 8 * 8, (a.SK + 7) / 8 * 8);
  a.G = std::max(1, std::min(a.P / a.SK, a.n_tiles));
  hipLaunchKernelGGL((gemm_kernel<DT, 5, false>), dim3(rg * a.P), block, 0, st, a);
  return hipGetLastError();
}

constexpr int MAX_SLICES = 16;   // gemm_slices() never exceeds this for K <= 32768

// Sum of the SK slice partials of elements (t, n..n+3), in slice order.  All
// loads are issued before the first add (no dependent round trips).
__device__ __forceinline__ float4 sum_slices4(const float* __restrict__ part, int SK, int T, int N,
                                              int t, int n) {
  float4 u[MAX_SLICES];
#pragma unroll
  for (int k = 0; k < MAX_SLICES; ++k)
    if (k < SK) u[k] = *reinterpret_cast<const float4*>(part + ((size_t)k * T + t) * N + n);
  float4 v = u[0];
#pragma unroll
  for (int k = 1; k < MAX_SLICES; ++k)
    if (k < SK) { v.x += u[k].x; v.y += u[k].y; v.z += u[k].z; v.w += u[k].w; }
  return v;
}

// Pack 8 consecutive values of row t starting at column col (col % 8 == 0)
// into the fragment layout: one 16-byte store for bf16, two for fp32.
template <int DT>
__device__ __forceinline__ void store8(void* xout, int t, int col, int S, const float* v) {
  if (DT == DT_BF16) {
    const uint4 u = make_uint4(f2bf_bits(v[0]) | (f2bf_bits(v[1]) << 16),
                               f2bf_bits(v[2]) | (f2bf_bits(v[3]) << 16),
                               f2bf_bits(v[4]) | (f2bf_bits(v[5]) << 16),
                               f2bf_bits(v[6]) | (f2bf_bits(v[7]) << 16));
    *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(xout) + frag_index<DT>(t, col, S)) = u;
  } else {
    float* f = reinterpret_cast<float*>(xout);
    *reinterpret_cast<float4*>(f + frag_index<DT>(t, col, S)) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(f + frag_index<DT>(t, col + 4, S)) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// Row scales of the split RMSNorm (see resid_kernel): chunk sums of h^2 per
// 1024-column chunk of a row.
constexpr int RES_THREADS = 128;               // 8 columns each
constexpr int RES_COLS = RES_THREADS * 8;      // columns per workgroup
constexpr int RES_MAX_PARTS = 8;               // chunks per row (d <= 8192)

// RMS scale of row t: 1 / sqrt(sum of its chunk sums, in chunk order, / d + eps).
// The row's chunk sums come with two 16-byte loads.
struct RowSsq {
  float4 a, b;   // chunk sums 0..7 of one row
};
__device__ __forceinline__ float row_scale_of(const RowSsq& r, int d, float eps) {
  static_assert(RES_MAX_PARTS == 8, "two 16-byte loads per row");
  const float c[RES_MAX_PARTS] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
  const int np = (d + RES_COLS - 1) / RES_COLS;
  float s = c[0];
#pragma unroll
  for (int i = 1; i < RES_MAX_PARTS; ++i)
    if (i < np) s += c[i];
  return 1.0f / sqrtf(s / (float)d + eps);
}
__device__ __forceinline__ float row_scale(const float* __restrict__ ssq, int t, int d, float eps) {
  const RowSsq r{reinterpret_cast<const float4*>(ssq + (size_t)t * RES_MAX_PARTS)[0],
                 reinterpret_cast<const float4*>(ssq + (size_t)t * RES_MAX_PARTS)[1]};
  return row_scale_of(r, d, eps);
}

// ------------------------------------------------------ gate/up + SwiGLU --
//
// For reductions of at most FK_MAX_S super-steps (d <= 4096 in bf16) the
// gate/up projection runs without K slices and applies SwiGLU itself:
//   * a workgroup owns pairs of tiles (gate features 16p .. 16p+15 and the up
//     features with the same indices) and reduces each over the whole of K:
//     wave w accumulates super-steps w, w+8, w+16, ... in order, the 8 wave
//     sums are added in wave order;
//   * its rows: up to 33, rows 0..31 as two register tiles and the 33rd from
//     LDS (one fragment column per super-step); blocks of more rows run as
//     32-row groups of one launch (the last group may hold 33), and with P a
//     multiple of 8 the groups that stream the same weights share an XCD;
//   * z = silu(gate) * up goes straight into the down projection's packed
//     activations: no slice partials, no separate SwiGLU launch.
// A row's arithmetic depends only on K, never on the block's rows.

constexpr int FK_MAX_S = 128;   // super-steps one workgroup reduces (16 per wave)
constexpr int FK_GROUP = 32;    // rows of a group held in registers

__host__ __device__ inline int fk_groups(int R) { return R <= FK_GROUP + 1 ? 1 : (R - 1 + FK_GROUP - 1) / FK_GROUP; }

__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.0f + expf(-g)) * u; }

struct FkArgs {
  const uint4* w;     // packed [2F, d]: gate rows, then up rows
  const uint4* x;     // packed activations of all R rows (h * gain of the FFN-side norm)
  void* z;            // packed [R, F] activations of the down projection
  int S, n_pairs;     // super-steps of d; F / 16
  int R, P, z_S;      // rows; workgroups per row group; super-steps of F
  const float* ssq;   // the norm's chunk sums of h^2 ([R][8]): row scales
  const float* ssqt;  // or (TS) its sums of h^2 per 16-column tile ([R][d / 16])
  int d;
  float eps;
};

// Row scales 1 / sqrt(sum h^2 / d + eps) of a row group from the per-tile sums
// of h^2 (ssqt[row][tile], d / 16 tiles of 16 columns; d a multiple of 256 and
// at most 4096), in a fixed order: a row's tile sums in chunks of 16 (one
// thread adds a chunk in tile order), then its chunk sums in chunk order.
// ts_issue requests the chunks of items threadIdx.x and threadIdx.x + 512
// (33 rows x 16 chunks at most); ts_chunks stores their sums to LDS; after a
// barrier, ts_rows turns each row's chunk sums into its scale.
constexpr int TS_CHUNKS = 16;   // chunks of a row, at most
struct TileSums {
  uint4 v[2][4];
};
__device__ __forceinline__ void ts_issue(TileSums& t, const float* ssqt, int R, int d, int row0, int T) {
  const int ntile = d / 16, nch = d / 256;
  const auto r = make_rsrc(ssqt, (unsigned)((size_t)R * ntile * 4));
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int item = (int)threadIdx.x + GEMM_WAVES * 64 * p, row = item / nch, ch = item - row * nch;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      t.v[p][q] = bload<0>(r, row < T ? (unsigned)(((size_t)(row0 + row) * ntile + ch * 16 + 4 * q) * 4) : OOB);
  }
}
__device__ __forceinline__ void ts_chunks(const TileSums& t, int d, int T, float (*tsc)[TS_CHUNKS]) {
  const int nch = d / 256;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int item = (int)threadIdx.x + GEMM_WAVES * 64 * p, row = item / nch, ch = item - row * nch;
    float s = __uint_as_float(t.v[p][0].x);
    s += __uint_as_float(t.v[p][0].y);
    s += __uint_as_float(t.v[p][0].z);
    s += __uint_as_float(t.v[p][0].w);
#pragma unroll
    for (int q = 1; q < 4; ++q) {
      s += __uint_as_float(t.v[p][q].x);
      s += __uint_as_float(t.v[p][q].y);
      s += __uint_as_float(t.v[p][q].z);
      s += __uint_as_float(t.v[p][q].w);
    }
    if (row < T) tsc[row][ch] = s;
  }
}
__device__ __forceinline__ void ts_rows(const float (*tsc)[TS_CHUNKS], int d, float eps, int T, float* rsl) {
  const int nch = d / 256, t = (int)threadIdx.x;
  if (t < T) {
    float s = tsc[t][0];
#pragma unroll
    for (int ch = 1; ch < TS_CHUNKS; ++ch)
      if (ch < nch) s += tsc[t][ch];
    rsl[t] = 1.0f / sqrtf(s / (float)d + eps);
  }
}

template <int DT, int MTV, int SPW, bool TS>
__global__ __launch_bounds__(GEMM_WAVES * 64) void gemm_swiglu_kernel(FkArgs a) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, c = lane & 15, grp = lane >> 4;
  const int rg = blockIdx.x / a.P, g = blockIdx.x - rg * a.P;
  const int ngroups = fk_groups(a.R);
  const int row0 = rg * FK_GROUP;
  const int T = rg == ngroups - 1 ? a.R - row0 : FK_GROUP;   // rows of this group, <= 33
  const bool rowl = MTV == 2 && T > 2 * 16;                  // the 33rd row, from LDS
  const int S = a.S;
  constexpr int NR = MTV == 2 ? 3 : 1;                       // reduced fragment tiles
  const auto xs = make_rsrc(a.x, (unsigned)((size_t)((a.R + 15) / 16) * S * 1024));
  const auto ws = make_rsrc(a.w, (unsigned)((size_t)2 * a.n_pairs * S * 1024));
  __shared__ uint4 rowx[MTV == 2 ? SPW * GEMM_WAVES * 4 : 1];   // [super-step][grp]: the 33rd row
  __shared__ f32x4 red[2][GEMM_WAVES][NR][64];
  // this thread's reduced item: fragment tile rm, lane rl (threads past NR * 64
  // repeat an item and store nothing)
  const int qq = threadIdx.x % (NR * 64);
  const bool qown = threadIdx.x < NR * 64;
  const int rm = qq >> 6, rl = qq & 63, rt = rm * 16 + (rl & 15);
  // the chunk sums (or tile sums) of the norm's row scale, requested first
  // (memory counters complete in order) and used only in the epilogue
  RowSsq rsq;
  TileSums tsum;
  __shared__ float rsl[TS ? FK_GROUP + 1 : 1];
  __shared__ float tsc[TS ? FK_GROUP + 1 : 1][TS_CHUNKS];
  if (!TS) {
    const auto sr = make_rsrc(a.ssq, (unsigned)((size_t)a.R * RES_MAX_PARTS * 4));
    const unsigned so = qown && rt < T ? (unsigned)((row0 + rt) * RES_MAX_PARTS * 4) : OOB;
    const uint4 u0 = bload<0>(sr, so), u1 = bload<0>(sr, so == OOB ? OOB : so + 16);
    rsq.a = make_float4(__uint_as_float(u0.x), __uint_as_float(u0.y), __uint_as_float(u0.z), __uint_as_float(u0.w));
    rsq.b = make_float4(__uint_as_float(u1.x), __uint_as_float(u1.y), __uint_as_float(u1.z), __uint_as_float(u1.w));
  } else {
    ts_issue(tsum, a.ssqt, a.R, a.d, row0, T);
  }
  uint4 xr[SPW][MTV];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int sl = wv + GEMM_WAVES * i;
#pragma unroll
    for (int m = 0; m < MTV; ++m)
      if (MTV == 2)   // (one register tile: requested with the first weights below)
        xr[i][m] = bload<0>(xs, (sl < S && m * 16 + c < min(T, 2 * 16))
                                    ? (unsigned)((((row0 / 16 + m) * S + sl) * 64 + lane) * 16) : OOB);
  }
  // the 33rd row: thread it holds entry it of rowx ([super-step][grp]; at most
  // one per thread, SPW <= 16); every entry the MFMAs read is written, zeros
  // past K or without a 33rd row
  static_assert(SPW * GEMM_WAVES * 4 <= GEMM_WAVES * 64, "one rowx entry per thread");
  const int it = threadIdx.x;
  const bool rowx_own = MTV == 2 && it < SPW * GEMM_WAVES * 4;
  const uint4 rowv = bload<0>(xs, (rowx_own && rowl && (it >> 2) < S)
                                      ? (unsigned)((((row0 / 16 + 2) * S + (it >> 2)) * 64 + (it & 3) * 16) * 16)
                                      : OOB);
  // tile k of this workgroup: pair g + (k / 2) P, gate (k even) or up (k odd)
  const int npair = g < a.n_pairs ? (a.n_pairs - g + a.P - 1) / a.P : 0;
  const int ntile = 2 * npair;
  auto tile_of = [&](int k) { return g + (k >> 1) * a.P + (k & 1) * a.n_pairs; };
  auto wload = [&](int k, int i) {
    const int sl = wv + GEMM_WAVES * i;
    return bload<2>(ws, (k < ntile && sl < S) ? (unsigned)(((tile_of(k) * S + sl) * 64 + lane) * 16) : OOB);
  };
  // the first half tile of weights is requested before the 33rd row is
  // stored: that store waits for every load issued before it (in order), so
  // the weight stream starts with the input loads instead of after them
  constexpr int HA = (SPW + 1) / 2, HB = SPW / 2;            // weight halves of a tile
  uint4 wa[HA], wb[HB > 0 ? HB : 1];
  if (MTV == 1) {
    // one register tile: inputs and the first half tile of weights requested
    // super-step by super-step, in the order the first MFMAs use them
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int sl = wv + GEMM_WAVES * i;
      xr[i][0] = bload<0>(xs, (sl < S && c < T) ? (unsigned)((((row0 / 16) * S + sl) * 64 + lane) * 16) : OOB);
      if (i < HA) wa[i] = wload(0, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < HA; ++i) wa[i] = wload(0, i);
  }
  if (rowx_own) rowx[it] = rowv;
  // (the tile sums were requested before the inputs: they are in by now)
  if (TS) ts_chunks(tsum, a.d, T, tsc);
  __syncthreads();
  if (TS) ts_rows(tsc, a.d, a.eps, T, rsl);   // (read after the first tile's barrier)
  f32x4 gate = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < ntile; ++k) {
    f32x4 acc[NR];
#pragma unroll
    for (int m = 0; m < NR; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the 33rd row's fragments are read from LDS RG super-steps at a time,
    // ahead of their MFMAs (one wait per group, not one per super-step)
    constexpr int RG = MTV == 2 ? 4 : (HA > 0 ? HA : 1);
    auto steps = [&](const uint4* wf, int i0, int n) {
#pragma unroll
      for (int g0 = 0; g0 < n; g0 += RG) {
        uint4 rv[RG];
#pragma unroll
        for (int j = 0; j < RG; ++j)
          if (MTV == 2 && g0 + j < n) {
            const uint4 r = rowx[(wv + GEMM_WAVES * (i0 + g0 + j)) * 4 + grp];
            rv[j] = c == 0 ? r : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
        for (int j = 0; j < RG; ++j)
          if (g0 + j < n) {
#pragma unroll
            for (int m = 0; m < MTV; ++m) acc[m] = mma<DT>(wf[g0 + j], xr[i0 + g0 + j][m], acc[m]);
            if (MTV == 2) acc[2] = mma<DT>(wf[g0 + j], rv[j], acc[2]);
          }
      }
    };
    // second half of this tile in flight while the first is multiplied, then
    // the first half of the next tile while the second is
#pragma unroll
    for (int i = 0; i < HB; ++i) wb[i] = wload(k, HA + i);
    steps(wa, 0, HA);
#pragma unroll
    for (int i = 0; i < HA; ++i) wa[i] = wload(k + 1, i);
    steps(wb, HA, HB);
    const int pb = k & 1;
#pragma unroll
    for (int m = 0; m < NR; ++m) red[pb][wv][m][lane] = acc[m];
    __syncthreads();
    f32x4 v = red[pb][0][rm][rl];
#pragma unroll
    for (int j = 1; j < GEMM_WAVES; ++j) v += red[pb][j][rm][rl];
    if (!(k & 1)) {
      gate = v;
    } else if (qown && rt < T) {
      // features 16p + 4(rl / 16) .. +3 of row row0 + rt
      const int f = 16 * (g + (k >> 1) * a.P) + 4 * (rl >> 4);
      const float rs = TS ? rsl[rt] : row_scale_of(rsq, a.d, a.eps);   // the norm's row scale
      float zv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) zv[r] = silu_mul(gate[r] * rs, v[r] * rs);
      const size_t fi = frag_index<DT>(row0 + rt, f, a.z_S);
      if (DT == DT_BF16) {
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.z) + fi) =
            make_uint2(f2bf_bits(zv[0]) | (f2bf_bits(zv[1]) << 16), f2bf_bits(zv[2]) | (f2bf_bits(zv[3]) << 16));
      } else {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.z) + fi) = make_float4(zv[0], zv[1], zv[2], zv[3]);
      }
    }
  }
}

template <int DT, int MTV, bool TS>
static void launch_gemm_swiglu(const FkArgs& a, int spw, dim3 grid, hipStream_t st) {
  const dim3 block(GEMM_WAVES * 64);
  switch (spw) {
    case 1: hipLaunchKernelGGL((gemm_swiglu_kernel<DT, MTV, 1, TS>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_swiglu_kernel<DT, MTV, 2, TS>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_swiglu_kernel<DT, MTV, 4, TS>), grid, block, 0, st, a); break;
    case 8: hipLaunchKernelGGL((gemm_swiglu_kernel<DT, MTV, 8, TS>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_swiglu_kernel<DT, MTV, 16, TS>), grid, block, 0, st, a); break;
  }
}

// z = silu(r x Wg^T) * (r x Wu^T) for R rows (r: each row's norm scale, from
// 1024-column chunk sums ssq, or from 16-column tile sums ssqt when given),
// when d / KS <= FK_MAX_S.
template <int DT>
static hipError_t gemm_swiglu(const uint4* wgu, const uint4* x, int F, int d, int R, void* z, const float* ssq,
                              const float* ssqt, float eps, hipStream_t st) {
  FkArgs a;
  a.w = wgu; a.x = x; a.z = z;
  a.ssq = ssq; a.ssqt = ssqt; a.d = d; a.eps = eps;
  if (ssqt && (d % 256 || d > 4096)) return hipErrorInvalidValue;
  a.S = d / Geo<DT>::KS;
  a.n_pairs = F / 16;
  a.R = R;
  a.z_S = F / Geo<DT>::KS;
  if (a.S > FK_MAX_S || F % 16) return hipErrorInvalidValue;
  int spw = 1;
  while (spw * GEMM_WAVES < a.S) spw *= 2;
  const int ng = fk_groups(R);
  // one row group: as many workgroups as give each the same count of pairs
  // (688 pairs: 230 x 3, not 176 x 3 + 80 x 2)
  const int per_wg = (a.n_pairs + 255) / 256;
  a.P = ng == 1 ? std::max(1, (a.n_pairs + per_wg - 1) / per_wg) : std::max(8, 256 / ng / 8 * 8);
  const dim3 grid(ng * a.P);
  if (ssqt) {
    if (R <= 16) launch_gemm_swiglu<DT, 1, true>(a, spw, grid, st);
    else launch_gemm_swiglu<DT, 2, true>(a, spw, grid, st);
  } else {
    if (R <= 16) launch_gemm_swiglu<DT, 1, false>(a, spw, grid, st);
    else launch_gemm_swiglu<DT, 2, false>(a, spw, grid, st);
  }
  return hipGetLastError();
}

inline bool fused_swiglu(int d, int dt) { return d / ks_of(dt) <= FK_MAX_S; }

// ------------------------------------------------ projection + epilogue --
//
// The QKV and O projections without K slices, the same loop as the gate/up
// kernel above (a workgroup reduces its tiles over the whole of K, rows 0..31
// in registers and the 33rd from LDS, 32-row groups for longer blocks), with
// the kernel that followed each of them folded into the epilogue:
//   * EP_ROPE (QKV): a workgroup owns pairs of tiles holding features i and
//     i + hd/2 of one head (tiles j and j + hd/32 of the head); the epilogue
//     applies the norm's row scale, rotates q and k at the row's position,
//     stores q and appends k and v to the row's KV-pool slot;
//   * EP_RESID (O): a workgroup owns single tiles; the epilogue adds the
//     projection to the residual stream, stores x = h * gain of the FFN-side
//     norm (the gate/up projection's packed input) and each row's sum of h^2
//     over the tile's 16 columns (the row scale's tile sums);
//   * EP_STORE (LM head): single tiles, the fp32 products stored as they are
//     (logits_kernel applies the final norm's row scale).
// Each output's reduction order depends only on K, never on the block's rows.

enum { EP_ROPE = 1, EP_RESID = 2, EP_STORE = 3 };

struct EpArgs {
  const uint4* w;        // packed weights [n_tiles][S][64]
  const uint4* x;        // packed activations of all R rows
  int S, n_tiles, n_items;   // super-steps of K; 16-feature tiles; pairs (ROPE) or tiles (RESID)
  int R, P;              // rows; workgroups per row group
  const float* ssq;      // ROPE: the input norm's 1024-column chunk sums [R][8]
  int d;                 // the norm's width
  float eps;
  // EP_ROPE
  int H, Hkv, hd;
  const int* pos;        // [R] rotary position of each row
  const float2* rope;    // [max_ctx][hd / 2] (cos, sin)
  const int* rowslot;    // [R] KV-pool slot
  void* q;               // [R][H][hd]
  void* kv_layer;        // this layer's KV pool (null: no K/V stores, for timing)
  void* kv_cap;          // test aid: the block's k and v rows, or null
  // EP_RESID
  float* h;              // [R][d] residual stream
  const float* gain;     // FFN-side norm gain [d]
  void* xout;            // packed [R][d] output x = h * gain
  int x_S;               // super-steps of d
  float* ssqt;           // [R][n_tiles] per-tile sums of h^2
  // EP_STORE
  float* y;              // [R][16 n_tiles] fp32 products
};

template <int DT, int MTV, int SPW, int EPI>
__global__ __launch_bounds__(GEMM_WAVES * 64) void gemm_ep_kernel(EpArgs a) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, c = lane & 15, grp = lane >> 4;
  const int rg = blockIdx.x / a.P, g = blockIdx.x - rg * a.P;
  const int ngroups = fk_groups(a.R);
  const int row0 = rg * FK_GROUP;
  const int T = rg == ngroups - 1 ? a.R - row0 : FK_GROUP;   // rows of this group, <= 33
  const bool rowl = MTV == 2 && T > 2 * 16;                  // the 33rd row, from LDS
  const int S = a.S;
  constexpr int NR = MTV == 2 ? 3 : 1;                       // reduced fragment tiles
  constexpr int ESZ = Geo<DT>::ESZ;
  const auto xs = make_rsrc(a.x, (unsigned)((size_t)((a.R + 15) / 16) * S * 1024));
  const auto ws = make_rsrc(a.w, (unsigned)((size_t)a.n_tiles * S * 1024));
  __shared__ uint4 rowx[MTV == 2 ? SPW * GEMM_WAVES * 4 : 1];   // [super-step][grp]: the 33rd row
  __shared__ f32x4 red[2][GEMM_WAVES][NR][64];
  const int qq = threadIdx.x % (NR * 64);
  const bool qown = threadIdx.x < NR * 64;
  const int rm = qq >> 6, rl = qq & 63, rt = rm * 16 + (rl & 15);
  const bool mine = qown && rt < T;                          // this thread stores row row0 + rt
  const int row = row0 + rt;
  // values used only in the epilogue, requested first: the rotary case's row
  // scale (chunk sums) and the group's positions and KV slots (kept in LDS,
  // as are the (cos, sin) of an item's features, so that the loop carries no
  // registers for them)
  RowSsq rsq;
  __shared__ int spos[EPI == EP_ROPE ? FK_GROUP + 1 : 1], sslot[EPI == EP_ROPE ? FK_GROUP + 1 : 1];
  __shared__ float2 scs[EPI == EP_ROPE ? FK_GROUP + 1 : 1][16];
  __shared__ float srs[EPI == EP_ROPE ? FK_GROUP + 1 : 1];
  int gpos = 0, gslot = 0;   // thread t < T: row row0 + t
  if (EPI == EP_ROPE) {
    const auto sr = make_rsrc(a.ssq, (unsigned)((size_t)a.R * RES_MAX_PARTS * 4));
    const unsigned so = mine ? (unsigned)(row * RES_MAX_PARTS * 4) : OOB;
    const uint4 u0 = bload<0>(sr, so), u1 = bload<0>(sr, so == OOB ? OOB : so + 16);
    rsq.a = make_float4(__uint_as_float(u0.x), __uint_as_float(u0.y), __uint_as_float(u0.z), __uint_as_float(u0.w));
    rsq.b = make_float4(__uint_as_float(u1.x), __uint_as_float(u1.y), __uint_as_float(u1.z), __uint_as_float(u1.w));
    const auto pr = make_rsrc(a.pos, (unsigned)(a.R * 4));
    const auto lr = make_rsrc(a.rowslot, (unsigned)(a.R * 4));
    const bool tr = (int)threadIdx.x < T;
    gpos = (int)__builtin_amdgcn_raw_buffer_load_b32(pr, tr ? (unsigned)((row0 + threadIdx.x) * 4) : OOB, 0, 0);
    gslot = (int)__builtin_amdgcn_raw_buffer_load_b32(lr, tr ? (unsigned)((row0 + threadIdx.x) * 4) : OOB, 0, 0);
  }
  uint4 xr[SPW][MTV];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int sl = wv + GEMM_WAVES * i;
#pragma unroll
    for (int m = 0; m < MTV; ++m)
      if (MTV == 2)
        xr[i][m] = bload<0>(xs, (sl < S && m * 16 + c < min(T, 2 * 16))
                                    ? (unsigned)((((row0 / 16 + m) * S + sl) * 64 + lane) * 16) : OOB);
  }
  static_assert(SPW * GEMM_WAVES * 4 <= GEMM_WAVES * 64, "one rowx entry per thread");
  const int it = threadIdx.x;
  const bool rowx_own = MTV == 2 && it < SPW * GEMM_WAVES * 4;
  const uint4 rowv = bload<0>(xs, (rowx_own && rowl && (it >> 2) < S)
                                      ? (unsigned)((((row0 / 16 + 2) * S + (it >> 2)) * 64 + (it & 3) * 16) * 16)
                                      : OOB);
  // items of this workgroup: g, g + P, ...; a pair is two tiles (k even: the
  // head's first half, k odd: its second half), a RESID item one tile
  constexpr int TPI = EPI == EP_ROPE ? 2 : 1;                // tiles per item
  const int nitem = g < a.n_items ? (a.n_items - g + a.P - 1) / a.P : 0;
  const int ntile = TPI * nitem;
  const int th = a.hd / 16, hp = th / 2;                     // tiles and pairs per head
  auto item_of = [&](int k) { return g + (k / TPI) * a.P; };
  auto tile_of = [&](int k) {
    if (EPI != EP_ROPE) return item_of(k);
    const int p = item_of(k);
    return (p / hp) * th + p % hp + (k & 1) * hp;
  };
  auto wload = [&](int k, int i) {
    const int sl = wv + GEMM_WAVES * i;
    return bload<2>(ws, (k < ntile && sl < S) ? (unsigned)(((tile_of(k) * S + sl) * 64 + lane) * 16) : OOB);
  };
  constexpr int HA = (SPW + 1) / 2, HB = SPW / 2;            // weight halves of a tile
  uint4 wa[HA], wb[HB > 0 ? HB : 1];
  if (MTV == 1) {
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      const int sl = wv + GEMM_WAVES * i;
      xr[i][0] = bload<0>(xs, (sl < S && c < T) ? (unsigned)((((row0 / 16) * S + sl) * 64 + lane) * 16) : OOB);
      if (i < HA) wa[i] = wload(0, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < HA; ++i) wa[i] = wload(0, i);
  }
  if (rowx_own) rowx[it] = rowv;
  // the input norm's row scales (their chunk sums were requested first: they
  // are in by now), positions and slots of the group's rows to LDS
  if (EPI == EP_ROPE) {
    if (mine && (rl >> 4) == 0) srs[rt] = row_scale_of(rsq, a.d, a.eps);
    if ((int)threadIdx.x < T) {
      spos[threadIdx.x] = gpos;
      sslot[threadIdx.x] = gslot;
    }
  }
  __syncthreads();
  f32x4 first = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < ntile; ++k) {
    // the epilogue's operands of this item, requested before its weights:
    // (cos, sin) of the thread's four features (ROPE), or the residual row
    // and gains of its four columns (RESID)
    uint4 ep0 = make_uint4(0u, 0u, 0u, 0u), ep1 = ep0;
    uint2 cs0 = make_uint2(0u, 0u), cs1 = cs0;   // ROPE: (cos, sin) of rows t / 16 and 32, feature t % 16
    if (k % TPI == 0) {
      const int f4 = 4 * (rl >> 4);
      if (EPI == EP_ROPE) {
        const int i0 = 16 * (item_of(k) % hp);                // the pair's first feature in the head
        const auto cr = make_rsrc(a.rope, (unsigned)0x7fffffff);
        const int r0 = (int)(threadIdx.x >> 4), j = (int)(threadIdx.x & 15);
        cs0 = bload64<0>(cr, r0 < T ? (unsigned)(((size_t)spos[r0] * (a.hd / 2) + i0 + j) * 8) : OOB);
        if (MTV == 2)
          cs1 = bload64<0>(cr, (threadIdx.x < 16 && T > 32) ? (unsigned)(((size_t)spos[32] * (a.hd / 2) + i0 + j) * 8)
                                                            : OOB);
      } else if (EPI == EP_RESID) {
        const int f = 16 * item_of(k) + f4;
        const auto hr = make_rsrc(a.h, (unsigned)((size_t)a.R * a.d * 4));
        const auto gr = make_rsrc(a.gain, (unsigned)(a.d * 4));
        ep0 = bload<0>(hr, mine ? (unsigned)(((size_t)row * a.d + f) * 4) : OOB);
        ep1 = bload<0>(gr, mine ? (unsigned)(f * 4) : OOB);
      }
    }
    f32x4 acc[NR];
#pragma unroll
    for (int m = 0; m < NR; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    constexpr int RG = MTV == 2 ? (EPI == EP_ROPE ? 2 : 4) : (HA > 0 ? HA : 1);   // (ROPE: fewer registers)
    auto steps = [&](const uint4* wf, int i0, int n) {
#pragma unroll
      for (int g0 = 0; g0 < n; g0 += RG) {
        uint4 rv[RG];
#pragma unroll
        for (int j = 0; j < RG; ++j)
          if (MTV == 2 && g0 + j < n) {
            const uint4 r = rowx[(wv + GEMM_WAVES * (i0 + g0 + j)) * 4 + grp];
            rv[j] = c == 0 ? r : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
        for (int j = 0; j < RG; ++j)
          if (g0 + j < n) {
#pragma unroll
            for (int m = 0; m < MTV; ++m) acc[m] = mma<DT>(wf[g0 + j], xr[i0 + g0 + j][m], acc[m]);
            if (MTV == 2) acc[2] = mma<DT>(wf[g0 + j], rv[j], acc[2]);
          }
      }
    };
#pragma unroll
    for (int i = 0; i < HB; ++i) wb[i] = wload(k, HA + i);
    steps(wa, 0, HA);
#pragma unroll
    for (int i = 0; i < HA; ++i) wa[i] = wload(k + 1, i);
    steps(wb, HA, HB);
    const int pb = k & 1;
#pragma unroll
    for (int m = 0; m < NR; ++m) red[pb][wv][m][lane] = acc[m];
    __syncthreads();
    f32x4 v = red[pb][0][rm][rl];
#pragma unroll
    for (int j = 1; j < GEMM_WAVES; ++j) v += red[pb][j][rm][rl];
    if (EPI == EP_ROPE && !(k & 1)) {
      // the item's (cos, sin) to LDS (read after the next barrier)
      first = v;
      const int r0 = (int)(threadIdx.x >> 4), j = (int)(threadIdx.x & 15);
      if (r0 < T) scs[r0][j] = make_float2(__uint_as_float(cs0.x), __uint_as_float(cs0.y));
      if (MTV == 2 && threadIdx.x < 16 && T > 32) scs[32][j] = make_float2(__uint_as_float(cs1.x), __uint_as_float(cs1.y));
    } else if (EPI == EP_ROPE && mine) {
      const int p = item_of(k), head = p / hp, f4 = 4 * (rl >> 4), i0 = 16 * (p % hp) + f4, half = a.hd / 2;
      const float rs = srs[rt];
      float cs[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float2 v2 = scs[rt][f4 + r];
        cs[2 * r] = v2.x;
        cs[2 * r + 1] = v2.y;
      }
      const int myslot = sslot[rt];
      float y1[4], y2[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x1 = first[r] * rs, x2 = v[r] * rs;
        if (head < a.H + a.Hkv) {
          y1[r] = fmaf(x1, cs[2 * r], -(x2 * cs[2 * r + 1]));   // (fixed contraction)
          y2[r] = fmaf(x2, cs[2 * r], x1 * cs[2 * r + 1]);
        } else {
          y1[r] = x1;
          y2[r] = x2;
        }
      }
      // stores through 32-bit buffer offsets (q, one KV-pool layer and the
      // capture stay below 2 GiB)
      auto put4 = [&](__amdgpu_buffer_rsrc_t r, unsigned e, const float* y) {
        if (DT == DT_BF16) {
          typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
          __builtin_amdgcn_raw_buffer_store_b64(
              u32x2{f2bf_bits(y[0]) | (f2bf_bits(y[1]) << 16), f2bf_bits(y[2]) | (f2bf_bits(y[3]) << 16)}, r,
              e * 2, 0, 0);
        } else {
          __builtin_amdgcn_raw_buffer_store_b128(
              u32x4{__float_as_uint(y[0]), __float_as_uint(y[1]), __float_as_uint(y[2]), __float_as_uint(y[3])}, r,
              e * 4, 0, 0);
        }
      };
      auto put1 = [&](__amdgpu_buffer_rsrc_t r, unsigned e, float y) {
        if (DT == DT_BF16)
          __builtin_amdgcn_raw_buffer_store_b16((uint16_t)f2bf_bits(y), r, e * 2, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), r, e * 4, 0, 0);
      };
      const unsigned layer_bytes = 0x7fffffffu;   // (the pool layer is below 2 GiB: checked at creation)
      const int page = myslot >> 6, sp = myslot & 63;
      // the row's address terms are formed here, not kept through the loop
      int row = row0 + rt;
      asm volatile("" : "+v"(row));
      if (head < a.H) {
        const auto qr = make_rsrc(a.q, (unsigned)((size_t)a.R * a.H * a.hd * ESZ));
        const unsigned qb = ((unsigned)row * a.H + head) * a.hd;
        put4(qr, qb + i0, y1);
        put4(qr, qb + i0 + half, y2);
      } else if (head < a.H + a.Hkv) {
        const int kh = head - a.H;
        if (a.kv_layer) {
          const auto kr = make_rsrc(a.kv_layer, layer_bytes);
          const unsigned kb = (((unsigned)page * 2 + 0) * a.Hkv + kh) * 64 * a.hd + (unsigned)sp * a.hd;
          put4(kr, kb + i0, y1);
          put4(kr, kb + i0 + half, y2);
        }
        if (a.kv_cap) {   // test aid: the block's k rows, [R][Hkv][hd]
          const auto cr = make_rsrc(a.kv_cap, (unsigned)((size_t)2 * a.R * a.Hkv * a.hd * ESZ));
          const unsigned cb = ((unsigned)row * a.Hkv + kh) * a.hd;
          put4(cr, cb + i0, y1);
          put4(cr, cb + i0 + half, y2);
        }
      } else {
        const int vh = head - a.H - a.Hkv;
        if (a.kv_layer) {
          const auto vr = make_rsrc(a.kv_layer, layer_bytes);
          const unsigned vb = (((unsigned)page * 2 + 1) * a.Hkv + vh) * 64 * a.hd;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            put1(vr, vb + (unsigned)(i0 + r) * 64 + sp, y1[r]);
            put1(vr, vb + (unsigned)(i0 + r + half) * 64 + sp, y2[r]);
          }
        }
        if (a.kv_cap) {   // test aid: the block's v rows after the k rows
          const auto cr = make_rsrc(a.kv_cap, (unsigned)((size_t)2 * a.R * a.Hkv * a.hd * ESZ));
          const unsigned cb = ((unsigned)a.R * a.Hkv + (unsigned)row * a.Hkv + vh) * a.hd;
          put4(cr, cb + i0, y1);
          put4(cr, cb + i0 + half, y2);
        }
      }
    } else if (EPI == EP_RESID) {
      // residual add, x = h * gain (bf16 for the next projection), and the
      // row's sum of h^2 over this tile's 16 columns (four lanes of 4 columns,
      // added by an xor butterfly: every lane gets the same value)
      const int tile = item_of(k), f = 16 * tile + 4 * (rl >> 4);
      const float hv[4] = {__uint_as_float(ep0.x), __uint_as_float(ep0.y), __uint_as_float(ep0.z),
                           __uint_as_float(ep0.w)};
      const float gn[4] = {__uint_as_float(ep1.x), __uint_as_float(ep1.y), __uint_as_float(ep1.z),
                           __uint_as_float(ep1.w)};
      float hn[4], xo[4], ss = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        hn[r] = hv[r] + v[r];
        ss = fmaf(hn[r], hn[r], ss);
        xo[r] = hn[r] * gn[r];
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      if (mine) {
        *reinterpret_cast<float4*>(a.h + (size_t)row * a.d + f) = make_float4(hn[0], hn[1], hn[2], hn[3]);
        const size_t fi = frag_index<DT>(row, f, a.x_S);
        if (DT == DT_BF16)
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.xout) + fi) =
              make_uint2(f2bf_bits(xo[0]) | (f2bf_bits(xo[1]) << 16), f2bf_bits(xo[2]) | (f2bf_bits(xo[3]) << 16));
        else
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.xout) + fi) = make_float4(xo[0], xo[1], xo[2], xo[3]);
        if ((rl >> 4) == 0) a.ssqt[(size_t)row * a.n_tiles + tile] = ss;
      }
    } else if (EPI == EP_STORE && mine) {
      const int f = 16 * item_of(k) + 4 * (rl >> 4);
      *reinterpret_cast<float4*>(a.y + (size_t)row * (16 * a.n_tiles) + f) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

template <int DT, int MTV, int EPI>
static void launch_gemm_ep(const EpArgs& a, int spw, dim3 grid, hipStream_t st) {
  const dim3 block(GEMM_WAVES * 64);
  switch (spw) {
    case 1: hipLaunchKernelGGL((gemm_ep_kernel<DT, MTV, 1, EPI>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_ep_kernel<DT, MTV, 2, EPI>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_ep_kernel<DT, MTV, 4, EPI>), grid, block, 0, st, a); break;
    case 8: hipLaunchKernelGGL((gemm_ep_kernel<DT, MTV, 8, EPI>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_ep_kernel<DT, MTV, 16, EPI>), grid, block, 0, st, a); break;
  }
}

// The projection of `a` (weights, activations, K = a.S super-steps, n_tiles,
// the epilogue's operands filled in) for R rows with epilogue EPI.
template <int DT, int EPI>
static hipError_t gemm_ep(EpArgs a, int R, hipStream_t st) {
  if (a.S > FK_MAX_S) return hipErrorInvalidValue;
  if (EPI == EP_ROPE && (a.hd % 32 || a.n_tiles % (a.hd / 16))) return hipErrorInvalidValue;
  a.R = R;
  int spw = 1;
  while (spw * GEMM_WAVES < a.S) spw *= 2;
  const int ng = fk_groups(R);
  a.P = ng == 1 ? std::max(1, std::min(256, a.n_items)) : std::max(8, 256 / ng / 8 * 8);
  const dim3 grid(ng * a.P);
  if (R <= 16) launch_gemm_ep<DT, 1, EPI>(a, spw, grid, st);
  else launch_gemm_ep<DT, 2, EPI>(a, spw, grid, st);
  return hipGetLastError();
}

// Whether the QKV and O projections run as gemm_ep_kernel (their reduction
// and the gate/up projection's fit one workgroup; rotary pairs of 16-feature
// tiles need head_dim a multiple of 32; the row scale's tile sums need d a
// multiple of 256 and at most 4096).  Depends only on the model's shape.
inline bool fused_proj(int d, int qdim, int hd, int dt) {
  return d / ks_of(dt) <= FK_MAX_S && qdim / ks_of(dt) <= FK_MAX_S && hd % 32 == 0 && d % 256 == 0 && d <= 4096;
}

// Whether the LM head runs as gemm_ep_kernel (EP_STORE) rather than with K
// slices: its reduction over d fits one workgroup.  Depends only on d.
inline bool lm_head_one_slice(int d, int dt) { return d / ks_of(dt) <= FK_MAX_S; }

// ------------------------------------------------------------ embed / norm --

// RMSNorm is split between this kernel and the consumers of the GEMM that
// follows it: here the residual stream of row t is updated (h = E[tok] in
// MODE 0, h += the GEMM slice partials in MODE 1), x = h * gain is stored,
// rounded to the model dtype, as the next GEMM's packed activations, and the
// sums of h^2 over the row's 1024-column chunks go to ssq[t][chunk]; the
// consumer multiplies every output of row t by r = 1 / sqrt(sum h^2 / d + eps)
// (row_scale), so RMSNorm(h) * gain * W = r * ((h * gain) W).  No workgroup
// needs a whole row: a row's work spreads over d / 1024 workgroups.  (The
// FFN-side norm of the fused path is instead formed in the O projection's
// epilogue, with sums of h^2 per 16-column tile: gemm_ep_kernel, ts_rows.)

template <int DT, int MODE>
__global__ __launch_bounds__(RES_THREADS) void resid_kernel(const void* __restrict__ embed,
                                                            const int* __restrict__ tok, float* __restrict__ h,
                                                            const float* __restrict__ part, int SK, int T,
                                                            const float* __restrict__ gain, int d,
                                                            void* __restrict__ xout, int x_S,
                                                            float* __restrict__ ssq) {
  __shared__ float sh[RES_THREADS / 64];
  const int t = blockIdx.y;
  const int col = (blockIdx.x * RES_THREADS + threadIdx.x) * 8;
  float ss = 0.f;
  if (col < d) {   // d % 8 == 0: a thread's 8 columns are all in range or all out
    float* hr = h + (size_t)t * d + col;
    float v[8];
    if (MODE == 0) {
      const size_t e0 = (size_t)tok[t] * d + col;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = load_elt<DT>(embed, e0 + e);
    } else {
      const float4 h0 = *reinterpret_cast<const float4*>(hr), h1 = *reinterpret_cast<const float4*>(hr + 4);
      const float4 p0 = sum_slices4(part, SK, T, d, t, col), p1 = sum_slices4(part, SK, T, d, t, col + 4);
      v[0] = h0.x + p0.x; v[1] = h0.y + p0.y; v[2] = h0.z + p0.z; v[3] = h0.w + p0.w;
      v[4] = h1.x + p1.x; v[5] = h1.y + p1.y; v[6] = h1.z + p1.z; v[7] = h1.w + p1.w;
    }
    const float4 g0 = *reinterpret_cast<const float4*>(gain + col), g1 = *reinterpret_cast<const float4*>(gain + col + 4);
    const float gn[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    *reinterpret_cast<float4*>(hr) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(hr + 4) = make_float4(v[4], v[5], v[6], v[7]);
    float o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      ss = fmaf(v[e], v[e], ss);
      o[e] = v[e] * gn[e];
    }
    store8<DT>(xout, t, col, x_S, o);
  }
  // fixed-order chunk sum: xor butterfly inside each wave, then the waves in order
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = ss;
  __syncthreads();
  if (threadIdx.x == 0) {
    float r = sh[0];
#pragma unroll
    for (int w = 1; w < RES_THREADS / 64; ++w) r += sh[w];
    ssq[t * RES_MAX_PARTS + blockIdx.x] = r;
  }
}


// q/k/v of row t from the QKV partials: rotary on q and k (pairs (i, i+hd/2)
// at the row's position), q to the block buffer, k and v into the row's KV
// pool slot (page * 64 + offset; V stored transposed per page).  One thread
// per pair.
template <int DT>
__global__ __launch_bounds__(256) void qkv_finish_kernel(const float* __restrict__ part, int SK, int T,
                                                         int N, int H, int Hkv, int hd,
                                                         const int* __restrict__ pos,
                                                         const float2* __restrict__ rope,
                                                         const int* __restrict__ rowslot,
                                                         void* __restrict__ q, void* __restrict__ kv_layer,
                                                         const float* __restrict__ ssq, int d, float eps,
                                                         void* __restrict__ kv_cap) {
  const int t = blockIdx.y;
  const int half = hd >> 1;
  const int pairs = (H + 2 * Hkv) * half;
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (p >= pairs) return;
  const int head = p / half, i = p % half;       // head over [q heads | k heads | v heads]
  const int f1 = head * hd + i, f2 = f1 + half;
  float p1[MAX_SLICES], p2[MAX_SLICES];
#pragma unroll
  for (int k = 0; k < MAX_SLICES; ++k)
    if (k < SK) {
      p1[k] = part[((size_t)k * T + t) * N + f1];
      p2[k] = part[((size_t)k * T + t) * N + f2];
    }
  float x1 = p1[0], x2 = p2[0];
#pragma unroll
  for (int k = 1; k < MAX_SLICES; ++k)
    if (k < SK) { x1 += p1[k]; x2 += p2[k]; }
  const float rs = row_scale(ssq, t, d, eps);   // the input norm's row scale
  x1 *= rs;
  x2 *= rs;
  const int slot = rowslot[t];
  const int page = slot >> 6, sp = slot & 63;
  if (head < H + Hkv) {
    const float2 cs = rope[(size_t)pos[t] * half + i];
    const float y1 = fmaf(x1, cs.x, -(x2 * cs.y));   // (fixed contraction)
    const float y2 = fmaf(x2, cs.x, x1 * cs.y);
    if (head < H) {
      const size_t qb = ((size_t)t * H + head) * hd;
      store_elt<DT>(q, qb + i, y1);
      store_elt<DT>(q, qb + i + half, y2);
    } else {
      const size_t kb = (((size_t)page * 2 + 0) * Hkv + (head - H)) * 64 * hd + (size_t)sp * hd;
      store_elt<DT>(kv_layer, kb + i, y1);
      store_elt<DT>(kv_layer, kb + i + half, y2);
      if (kv_cap) {   // test aid: the block's k rows, [T][Hkv][hd]
        const size_t cb = ((size_t)t * Hkv + (head - H)) * hd;
        store_elt<DT>(kv_cap, cb + i, y1);
        store_elt<DT>(kv_cap, cb + i + half, y2);
      }
    }
  } else {
    const size_t vb = (((size_t)page * 2 + 1) * Hkv + (head - H - Hkv)) * 64 * hd;
    store_elt<DT>(kv_layer, vb + (size_t)i * 64 + sp, x1);
    store_elt<DT>(kv_layer, vb + (size_t)(i + half) * 64 + sp, x2);
    if (kv_cap) {     // test aid: the block's v rows after the k rows
      const size_t cb = ((size_t)T * Hkv + (size_t)t * Hkv + (head - H - Hkv)) * hd;
      store_elt<DT>(kv_cap, cb + i, x1);
      store_elt<DT>(kv_cap, cb + i + half, x2);
    }
  }
}

// z = silu(gate) * up from the gate/up partials (rows [0, F) gate, [F, 2F)
// up), packed as the down projection's activations.  8 features per thread.
template <int DT>
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ part, int SK, int T, int F,
                                                     void* __restrict__ zout, int z_S,
                                                     const float* __restrict__ ssq, int d, float eps) {
  const int t = blockIdx.y;
  const int ch = blockIdx.x * 256 + threadIdx.x;
  if (ch * 8 >= F) return;
  const int f = ch * 8, N = 2 * F;
  const float4 g0 = sum_slices4(part, SK, T, N, t, f), g1 = sum_slices4(part, SK, T, N, t, f + 4);
  const float4 u0 = sum_slices4(part, SK, T, N, t, F + f), u1 = sum_slices4(part, SK, T, N, t, F + f + 4);
  const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float u[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
  float z[8];
  const float rs = row_scale(ssq, t, d, eps);   // the input norm's row scale
#pragma unroll
  for (int e = 0; e < 8; ++e) z[e] = silu_mul(g[e] * rs, u[e] * rs);
  store8<DT>(zout, t, f, z_S, z);
}

// Logits of row t from the LM-head partials, plus the (value, -index) maximum
// of each 2048-column chunk.
__device__ __forceinline__ unsigned long long amax_key(float v, int idx) {
  uint32_t u = __float_as_uint(v);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0ull;   // NaN never wins
  if ((u & 0x7fffffffu) == 0) u = 0;                   // -0 ties with +0
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((unsigned long long)ord << 32) | (0xffffffffu - (uint32_t)idx);
}

// Descending compare-exchange of two keys.
__device__ __forceinline__ void cx_desc(unsigned long long& a, unsigned long long& b) {
  const unsigned long long hi = a > b ? a : b, lo = a > b ? b : a;
  a = hi;
  b = lo;
}

// Sort 8 keys into descending order (Batcher's odd-even merge network).
__device__ __forceinline__ void sort8_desc(unsigned long long (&k)[8]) {
  cx_desc(k[0], k[1]); cx_desc(k[2], k[3]); cx_desc(k[4], k[5]); cx_desc(k[6], k[7]);
  cx_desc(k[0], k[2]); cx_desc(k[1], k[3]); cx_desc(k[4], k[6]); cx_desc(k[5], k[7]);
  cx_desc(k[1], k[2]); cx_desc(k[5], k[6]);
  cx_desc(k[0], k[4]); cx_desc(k[1], k[5]); cx_desc(k[2], k[6]); cx_desc(k[3], k[7]);
  cx_desc(k[2], k[4]); cx_desc(k[3], k[5]);
  cx_desc(k[1], k[2]); cx_desc(k[3], k[4]); cx_desc(k[5], k[6]);
}

// The 8 largest keys held by a wave whose lanes each hold a descending list
// of 8.  Keys are distinct (the column index is part of the key) except 0,
// which stands for "no element"; every lane receives the same result.
__device__ __forceinline__ void wave_top8(unsigned long long (&k)[8], unsigned long long (&out)[8]) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    unsigned long long m = k[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const unsigned long long x = __shfl_xor(m, o);
      m = x > m ? x : m;
    }
    out[r] = m;
    const bool pop = m != 0ull && k[0] == m;
#pragma unroll
    for (int i = 0; i < 7; ++i) k[i] = pop ? k[i + 1] : k[i];
    k[7] = pop ? 0ull : k[7];
  }
}

// Logits of row t from the LM-head partials (times the final norm's row
// scale), plus, per 2048-column chunk,
// either the largest key (TOPK false: amax[t][chunk]) or the 8 largest keys
// in descending order (TOPK true: amax[t][chunk][8]).
template <bool TOPK>
__global__ __launch_bounds__(256) void logits_kernel(const float* __restrict__ part, int SK, int T, int V,
                                                     float* __restrict__ logits,
                                                     unsigned long long* __restrict__ amax, int nchunk,
                                                     const float* __restrict__ ssq, int d, float eps) {
  const int t = blockIdx.y;
  const int col = (blockIdx.x * 256 + threadIdx.x) * 8;
  unsigned long long key[8] = {0ull, 0ull, 0ull, 0ull, 0ull, 0ull, 0ull, 0ull};
  if (col < V) {   // V is a multiple of 16: a thread's 8 columns are all in range or all out
    const float rs = row_scale(ssq, t, d, eps);   // the final norm's row scale
    float4 a = sum_slices4(part, SK, T, V, t, col), b = sum_slices4(part, SK, T, V, t, col + 4);
    a.x *= rs; a.y *= rs; a.z *= rs; a.w *= rs;
    b.x *= rs; b.y *= rs; b.z *= rs; b.w *= rs;
    float* lr = logits + (size_t)t * V + col;
    *reinterpret_cast<float4*>(lr) = a;
    *reinterpret_cast<float4*>(lr + 4) = b;
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) key[e] = amax_key(v[e], col + e);
  }
  if constexpr (!TOPK) {
    __shared__ unsigned long long sh[256];
    unsigned long long best = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) best = key[e] > best ? key[e] : best;
    sh[threadIdx.x] = best;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w && sh[threadIdx.x + w] > sh[threadIdx.x]) sh[threadIdx.x] = sh[threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) amax[(size_t)t * nchunk + blockIdx.x] = sh[0];
  } else {
    __shared__ unsigned long long sh[4][8];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    unsigned long long top[8];
    sort8_desc(key);
    wave_top8(key, top);
    if (lane == 0) {
#pragma unroll
      for (int i = 0; i < 8; ++i) sh[wv][i] = top[i];
    }
    __syncthreads();
    if (wv == 0) {
#pragma unroll
      for (int i = 0; i < 8; ++i) key[i] = lane < 4 ? sh[lane & 3][i] : 0ull;
      wave_top8(key, top);
      unsigned long long mine = 0ull;
#pragma unroll
      for (int i = 0; i < 8; ++i) mine = lane == i ? top[i] : mine;
      if (lane < 8) amax[((size_t)t * nchunk + blockIdx.x) * 8 + lane] = mine;
    }
  }
}

// --------------------------------------------------------------- attention --

struct AttnArgs {
  const void* q;            // [T][H][hd]
  const void* kv_layer;     // [pages][2][Hkv][64*hd]
  const int* ptable;        // [B][ptable_len]
  const int* pos;
  const unsigned char* path;  // tree: [B*T][64], entry j-1 = block row at depth j on row t's path
  const int* info;          // [B][4]: committed positions n, splits in use
  int T, H, Hkv, G, ncols;  // T rows and ncols = T * G query columns per sequence
  int B;                    // sequences: rows b*T .. b*T + T - 1, columns b*ncols ..
  int tree;
  // 0: every split of the grid; 1: only splits holding committed keys and the
  // pending row alone (sp < (n + 1) / SPLIT; what every row of a draft tree
  // sees unmasked); 2: the splits from (n + 1) / SPLIT on, grid y counted
  // from there (a tree's own rows)
  int split_mode;
  float scale_log2;         // log2(e) / sqrt(hd)
  float* part;              // [splits][Hkv][B * ncols][hd + 2]
  int max_pages;            // pages per layer in the pool
  int ptable_len;           // page-table entries (multiple of 4, 16-byte aligned)
};

constexpr int SPLIT = 256;   // keys per split (4 sub-tiles of 64)
constexpr int NSUB = SPLIT / 64;


// workgroup size: 16 waves (4 query tiles x 4 sub-tiles); the tree variant
// runs 8 waves (2 query tiles) so that its gather loop has 256 registers
constexpr int att_threads(bool tree) { return tree ? 512 : 1024; }
constexpr int att_qt(bool tree) { return att_threads(tree) / 64 / NSUB; }

// LDS image of one split: K rows [NSUB][64][HD] and V^T [NSUB][HD][64], rows
// padded by 16 bytes to spread banks.
// Position, within a bf16 V^T row of the LDS image, of the value of sub-tile
// key k (0..63).  A PV step's B operand takes keys 32j + 4grp + 0..3 and
// 32j + 16 + 4grp + 0..3 in MFMA order (the order of the score fragments);
// storing them side by side lets a lane fetch its value fragment with one
// 16-byte read, which with the 144-byte row pitch also hits 32 distinct banks
// per 8 lanes (two 8-byte reads conflicted two-way).  fp32 rows keep key order.
__host__ __device__ constexpr int vt_pos(int k) {
  return 32 * (k >> 5) + 8 * ((k >> 2) & 3) + 4 * ((k >> 4) & 1) + (k & 3);
}

template <int DT, int HD, int THREADS> struct AttnLds {
  static constexpr int ESZ = Geo<DT>::ESZ;
  static constexpr int ROWB = HD * ESZ, KROW = ROWB + 16, VROW = 64 * ESZ + 16;
  static constexpr int KSUB = 64 * KROW, VSUB = HD * VROW;
  static constexpr int KV_BYTES = NSUB * (KSUB + VSUB);
  static constexpr int ST_BYTES = (THREADS / 64) * (16 * (HD + 4) + 32) * 4;   // merge states
  static constexpr int BYTES = KV_BYTES > ST_BYTES ? KV_BYTES : ST_BYTES;
  static constexpr int UNITS = 2 * 64 * HD * ESZ / 16;             // uint4 per sub-tile (K + V)
  static constexpr int PER = (NSUB * UNITS + THREADS - 1) / THREADS;
};

// Scores of the sub-tile, S^T = K Q^T (head-dim step outermost, so
// consecutive MFMAs feed independent accumulators), scaled to log2 units,
// with keys past the column's position set to -inf; m = their maximum.
template <int DT, int HD, class KFn>
__device__ __forceinline__ void subtile_scores(const uint4 (&qf)[HD / Geo<DT>::KS], KFn kfn, int base, int mypos,
                                               float scale_log2, int grp, f32x4 (&sacc)[4], float& m) {
  constexpr int NS = HD / Geo<DT>::KS;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) sacc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    uint4 kf[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) kf[kt] = kfn(kt, s);
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) sacc[kt] = mma<DT>(kf[kt], qf[s], sacc[kt]);
  }
  m = -INFINITY;
  // a sub-tile that every column of the wave sees whole (columns past the
  // block, position -1, hold nothing that is kept) skips the position test:
  // the same values as with it
  if (__all(mypos < 0 || base + 63 <= mypos)) {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = sacc[kt][r] * scale_log2;
        sacc[kt][r] = x;
        m = fmaxf(m, x);
      }
  } else {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kp = base + 16 * kt + 4 * grp + r;
        const float x = kp <= mypos ? sacc[kt][r] * scale_log2 : -INFINITY;
        sacc[kt][r] = x;
        m = fmaxf(m, x);
      }
  }
  m = xmax16(m);
  m = xmax32(m);
}

// From the scores and their maximum m: l = sum 2^(s-m) and o += sum 2^(s-m) v
// (columns with own == false add exact zeros to o).
template <int DT, int HD, bool STREAMV, class VFn, class VPrep>
__device__ __forceinline__ void subtile_values(f32x4 (&sacc)[4], float m, VFn vfn, VPrep vprep, int grp, bool own,
                                               float& l, f32x4 (&o)[HD / 16]) {
  constexpr int ND = HD / 16;
  (void)grp;
  const float m_use = m != -INFINITY ? m : 0.f;
  l = 0.f;
#pragma unroll
  for (int kt = 0; kt < 4; ++kt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // v_exp_f32: exp2(-inf) = 0 for hidden keys; a weight below 2^-126
      // (a score 126 below the maximum) is 0 rather than a denormal
      const float pv = __builtin_amdgcn_exp2f(sacc[kt][r] - m_use);
      sacc[kt][r] = own ? pv : 0.f;
      l += pv;
    }
  l = xsum16(l);
  l = xsum32(l);
  // O^T = V^T P^T over the sub-tile's 64 keys
  if (DT == DT_BF16) {
    // P enters the bf16 MFMA as hi + lo bf16 parts (about 16 significant
    // bits), so the weights of the value rows keep near-fp32 precision.
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      vprep(k2);
      uint32_t ph[4], pl[4];   // packed pairs: elements 2h (low) and 2h + 1
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float pa = sacc[2 * k2 + (h >> 1)][2 * (h & 1)], pb = sacc[2 * k2 + (h >> 1)][2 * (h & 1) + 1];
        ph[h] = bf16x2_bits(pa, pb);
        pl[h] = bf16x2_bits(pa - __uint_as_float(ph[h] << 16), pb - __uint_as_float(ph[h] & 0xffff0000u));
      }
      const uint4 pfh = make_uint4(ph[0], ph[1], ph[2], ph[3]);
      const uint4 pfl = make_uint4(pl[0], pl[1], pl[2], pl[3]);
      if (STREAMV) {
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
          const uint4 vf = vfn(dt, k2);
          o[dt] = mma<DT>(vf, pfh, o[dt]);
          o[dt] = mma<DT>(vf, pfl, o[dt]);
        }
      } else {
        uint4 vf[ND];
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) vf[dt] = vfn(dt, k2);
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) o[dt] = mma<DT>(vf[dt], pfh, o[dt]);
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) o[dt] = mma<DT>(vf[dt], pfl, o[dt]);
      }
    }
  } else {
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      vprep(kt);
      const uint4 pf = make_uint4(__float_as_uint(sacc[kt][0]), __float_as_uint(sacc[kt][1]),
                                  __float_as_uint(sacc[kt][2]), __float_as_uint(sacc[kt][3]));
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) o[dt] = mma<DT>(vfn(dt, kt), pf, o[dt]);
    }
  }
}

// One 64-key sub-tile for the wave's 16 query columns: scores S^T = K Q^T
// (head-dim step outermost, so consecutive MFMAs feed independent
// accumulators), m = max visible scaled score, l = sum 2^(s-m) and
// o = sum 2^(s-m) v.  kfn(kt, s) gives the key fragment of key 16kt + c at head
// dims s*KS + grp*EPL ..; vfn(dt, j) the value fragment of output dims 16dt + c
// (bf16, j = k2: keys 32j + 4grp + 0..3 then 32j + 16 + 4grp + 0..3; fp32,
// j = kt: keys 16j + 4grp + 0..3).  Key 16kt + 4grp + r of the sub-tile sits at
// position base + 16kt + 4grp + r and is visible to a column iff that position
// is <= the column's own.  A column's result depends only on its query, the
// key/value data and the positions, never on the other columns.  o is
// accumulated into (the caller clears it); columns with own == false add
// exact zeros to it.  vprep(j) runs before the value fragments of PV step j
// (k2 or kt) are fetched.  STREAMV fetches each value fragment right before
// its MFMAs (fewer live registers; the same arithmetic in the same order).
template <int DT, int HD, bool STREAMV, class KFn, class VFn, class VPrep>
__device__ __forceinline__ void subtile_state(const uint4 (&qf)[HD / Geo<DT>::KS], KFn kfn, VFn vfn, VPrep vprep,
                                              int base, int mypos, float scale_log2, int grp, bool own,
                                              float& m, float& l, f32x4 (&o)[HD / 16]) {
  f32x4 sacc[4];
  subtile_scores<DT, HD>(qf, kfn, base, mypos, scale_log2, grp, sacc, m);
  subtile_values<DT, HD, STREAMV>(sacc, m, vfn, vprep, grp, own, l, o);
}

// Stage sub-tiles 0 .. nsub-1 of the split starting at position base0 (K rows
// and V^T, KV head gkv) in LDS with one batch of loads per thread; slots at or
// past nkeys (not yet written) read as zeros.
// The NSUB page numbers of the split starting at position base0, with one
// vector load (scalar loads of the uniform addresses would each wait for the
// previous one); entries past the table read as 0.
__device__ __forceinline__ uint4 split_pages(const AttnArgs& a, const int* ptable, int base0) {
  static_assert(NSUB == 4, "one 16-byte load of page numbers");
  return bload<0>(make_rsrc(ptable, (unsigned)(a.ptable_len * 4)), (unsigned)((base0 >> 6) * 4));
}

template <int DT, int HD, int THREADS>
__device__ __forceinline__ void stage_split(const AttnArgs& a, const uint4 p4, int gkv, int base0, int nsub,
                                            int nkeys, unsigned char* lds) {
  using LY = AttnLds<DT, HD, THREADS>;
  constexpr int ESZ = Geo<DT>::ESZ;
  constexpr int ROWB = LY::ROWB, KROW = LY::KROW, VROW = LY::VROW;
  const size_t layer_bytes = (size_t)a.max_pages * 2 * a.Hkv * 64 * HD * ESZ;
  const auto rs = make_rsrc(a.kv_layer, (unsigned)layer_bytes);
  constexpr int HALF = LY::UNITS / 2;                  // uint4 per K (or V) sub-tile
  // the split's NSUB page numbers (split_pages)
  int pg[NSUB];
  pg[0] = (int)p4.x; pg[1] = (int)p4.y; pg[2] = (int)p4.z; pg[3] = (int)p4.w;
  uint4 tmp[LY::PER];
  unsigned dst[LY::PER];
#pragma unroll
  for (int j = 0; j < LY::PER; ++j) {
    const int idx = threadIdx.x + j * THREADS;
    const int st = idx / LY::UNITS, rem = idx % LY::UNITS;
    const int kv = rem / HALF, u = rem % HALF;
    unsigned off = OOB;
    dst[j] = 0xffffffffu;
    if (st < nsub) {
      const int base = base0 + st * 64;
      int page = pg[0];
#pragma unroll
      for (int q = 1; q < NSUB; ++q) page = st == q ? pg[q] : page;
      const int valid = nkeys - base;
      off = (unsigned)(((((size_t)page * 2 + kv) * a.Hkv + gkv) * 64 * HD) * ESZ + (size_t)u * 16);
      if (kv == 0) {
        const int row = u / (ROWB / 16), col = u % (ROWB / 16);
        if (row >= valid) off = OOB;                    // unwritten slots read as zeros
        dst[j] = st * LY::KSUB + row * KROW + col * 16;
      } else {
        constexpr int VU = 64 * ESZ / 16;               // uint4 per V^T row
        dst[j] = NSUB * LY::KSUB + st * LY::VSUB + (u / VU) * VROW + (u % VU) * 16;
        dst[j] |= (unsigned)min(valid, 64) << 24;       // remember the valid key count
      }
    }
    tmp[j] = bload<0>(rs, off);
  }
#pragma unroll
  for (int j = 0; j < LY::PER; ++j) {
    if (dst[j] == 0xffffffffu) continue;
    unsigned d = dst[j];
    uint4 v = tmp[j];
    if ((d >> 24) != 0) {
      // V^T chunk: zero the key columns of unwritten slots
      const int valid = (int)(d >> 24);
      d &= 0x00ffffffu;
      if (valid < 64) {
        const int col0 = (((d - NSUB * LY::KSUB) % LY::VSUB) % VROW) / ESZ;
        uint32_t w4[4] = {v.x, v.y, v.z, v.w};
        if (DT == DT_BF16) {
          for (int e = 0; e < 8; ++e)
            if (col0 + e >= valid) w4[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
        } else {
          for (int e = 0; e < 4; ++e)
            if (col0 + e >= valid) w4[e] = 0;
        }
        v = make_uint4(w4[0], w4[1], w4[2], w4[3]);
      }
      if (DT == DT_BF16) {
        // keys col0 .. col0 + 3 and col0 + 4 .. col0 + 7 to their places
        const int col0 = (((d - NSUB * LY::KSUB) % LY::VSUB) % VROW) / ESZ;
        unsigned char* row = lds + d - col0 * ESZ;
        *reinterpret_cast<uint2*>(row + vt_pos(col0) * ESZ) = make_uint2(v.x, v.y);
        *reinterpret_cast<uint2*>(row + vt_pos(col0 + 4) * ESZ) = make_uint2(v.z, v.w);
        continue;
      }
    }
    *reinterpret_cast<uint4*>(lds + d) = v;
  }
  }

// Split attention.  Workgroup (KV head g, split sp, query-tile group) stages
// the split's keys and values (positions sp*256 .. sp*256+255, four 64-key
// sub-tiles) in LDS with one batch of loads; each wave then takes one tile of
// 16 query columns (query heads of group g x block rows) and computes, over
// the whole split, m = max scaled score, l = sum 2^(s-m) and o = sum 2^(s-m) v
// in a fixed order (sub-tile, key tile, key), stored for attn_combine_kernel.
// A column's arithmetic depends only on the key positions, never on T or on
// which workgroup ran it; keys it cannot see contribute exact zeros.
// (the body of one workgroup, block (bx, by, bz) of the grid described
// above, with its LDS at lds: AttnLds<DT, HD, att_threads(TREE)>::BYTES)
template <int DT, int HD, bool TREE>
__device__ __forceinline__ void attn_block(AttnArgs a, int bx, int by, int bz, unsigned char* lds) {
  constexpr int ATT_THREADS = att_threads(TREE), ATT_QT = att_qt(TREE);
  using LY = AttnLds<DT, HD, ATT_THREADS>;
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL, ESZ = Geo<DT>::ESZ;
  constexpr int NS = HD / KS;          // fragments along head_dim
  constexpr int ND = HD / 16;          // output dim tiles
  constexpr int ROWB = LY::ROWB, KROW = LY::KROW, VROW = LY::VROW;
  unsigned char* Kall = lds;
  unsigned char* Vall = lds + NSUB * LY::KSUB;

  const int nqt = (a.ncols + 15) / 16;
  const int qgs = (nqt + ATT_QT - 1) / ATT_QT;   // query-tile groups per sequence
  const int gkv = bx, b = bz / qgs, qgrp = bz % qgs;
  int sp = by;
  // this sequence's rows, positions, paths, pages and step state
  const int rb = b * a.T;
  const int* pos = a.pos + rb;
  const unsigned char* path = a.path + (size_t)rb * 64;
  const int* ptable = a.ptable + b * a.ptable_len;
  // (n, splits in use) with one vector load, and the split's page numbers
  // in the same round trip where the split does not depend on n
  const uint2 inf = bload64<0>(make_rsrc(a.info + 4 * b, 8), 0);
  uint4 p4 = a.split_mode != 2 ? split_pages(a, ptable, sp * SPLIT) : make_uint4(0u, 0u, 0u, 0u);
  const int n = __builtin_amdgcn_readfirstlane((int)inf.x);
  if (a.split_mode == 2) {
    sp += (n + 1) / SPLIT;
    p4 = split_pages(a, ptable, sp * SPLIT);
  }
  if (sp >= __builtin_amdgcn_readfirstlane((int)inf.y)) return;   // the grid covers the longest context
  if (a.split_mode == 1 && sp >= (n + 1) / SPLIT) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int grp = lane >> 4, c = lane & 15;
  const int nkeys = n + a.T;            // slots written so far
  const int base0 = sp * SPLIT;
  const int nsub = min(NSUB, (nkeys - base0 + 63) / 64);

  // wave -> (query tile of this workgroup, sub-tile of the split); the query
  // fragments (B operand: column qc, head dims s*KS + grp*EPL ..) are fetched
  // together with the staging loads
  const int qi = wv / NSUB, st = wv % NSUB;
  const int qt = qgrp * ATT_QT + qi;
  const bool work = qt < nqt && st < nsub;     // uniform per wave
  const int qc = qt * 16 + c;
  const bool colok = qc < a.ncols;
  const int t = colok ? qc / a.G : 0;
  const int head = gkv * a.G + (colok ? qc % a.G : 0);
  const int mypos = colok ? pos[t] : -1;
  const int base = base0 + st * 64;
  uint4 qf[NS];
  {
  const auto qr = make_rsrc(a.q, (unsigned)((size_t)a.B * a.T * a.H * ROWB));
  const unsigned qb = (unsigned)(((size_t)(rb + t) * a.H + head) * ROWB);
  // (tree: waves past the staged sub-tiles may gather, so every wave of a
  // live query tile needs its queries)
  const bool need = TREE ? qt < nqt : work;
#pragma unroll
  for (int s = 0; s < NS; ++s) qf[s] = bload<0>(qr, (need && colok) ? qb + (unsigned)((s * KS + grp * EPL) * ESZ) : OOB);
  }

  // ---- stage every sub-tile of the split with one batch of loads ----
  stage_split<DT, HD, ATT_THREADS>(a, p4, gkv, base0, nsub, nkeys, lds);
  __syncthreads();

  // A tree row at depth j sits at position n + j and sees, at positions
  // n+1 .. n+j, its ancestors in depth order: exactly what the chain along its
  // path would hold there.  Sub-tiles reaching those positions ("gather"
  // sub-tiles g0..g1 of the query tile) are computed once per block row, from
  // keys and values gathered by position; the rows of the tile are dealt out
  // to its NSUB waves.  Every other sub-tile holds committed keys and the
  // pending row only, the same for every row, and is read from the staged
  // image as in the linear case.  The waves of sub-tiles g0 .. NSUB-1 do the
  // gathering (sub-tiles past g1 lie beyond every row of the tile: their state
  // is empty), each serving one gather sub-tile and a share of the rows.
  int g0 = 0, g1 = -1;
  if (TREE) {
  int mx = mypos;
  mx = max(mx, __shfl_xor(mx, 1));
  mx = max(mx, __shfl_xor(mx, 2));
  mx = max(mx, __shfl_xor(mx, 4));
  mx = max(mx, __shfl_xor(mx, 8));   // uniform: the query tile's largest position
  if (mx > n && mx >= base0) {
    g0 = n + 1 >= base0 ? (n + 1 - base0) >> 6 : 0;
    g1 = min(nsub - 1, (mx - base0) >> 6);
  }
  }
  const bool worker = TREE && g1 >= g0 && st >= g0;

  float m = -INFINITY, l = 0.f;
  f32x4 o[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (work && !worker) {
  const unsigned char* Ks = Kall + st * LY::KSUB;
  const unsigned char* Vt = Vall + st * LY::VSUB;
  auto kfn = [&](int kt, int s) {
    return *reinterpret_cast<const uint4*>(Ks + (size_t)(16 * kt + c) * KROW + (s * KS + grp * EPL) * ESZ);
  };
  auto vfn = [&](int dt, int j) {
    const unsigned char* vr = Vt + (size_t)(16 * dt + c) * VROW;
    if (DT == DT_BF16) return *reinterpret_cast<const uint4*>(vr + (32 * j + 8 * grp) * ESZ);   // (vt_pos)
    return *reinterpret_cast<const uint4*>(vr + (16 * j + 4 * grp) * ESZ);
  };
  subtile_state<DT, HD, false>(qf, kfn, vfn, [](int) {}, base, mypos, a.scale_log2, grp, true, m, l, o);
  }

  // a gathering wave serves sub-tile g0 + gi (positions n+1 .. n+64 span at
  // most two sub-tiles) and its rows t_lo + kk, t_lo + kk + nw, ... (kk-th of
  // the nw waves serving that sub-tile), accumulating in o
  const int t_lo = (qt * 16) / a.G, t_hi = (min(qt * 16 + 15, a.ncols - 1)) / a.G;
  const int ng = g1 - g0 + 1, wk = st - g0;
  const int gi = worker ? wk % ng : 0, kk = worker ? wk / ng : 0;
  const int nw = worker ? (NSUB - g0 - gi + ng - 1) / ng : 1;
  if (worker && qt < nqt && t_lo + kk <= t_hi) {
  const size_t layer_bytes = (size_t)a.max_pages * 2 * a.Hkv * 64 * HD * ESZ;
  const auto rs = make_rsrc(a.kv_layer, (unsigned)layer_bytes);
  // Gathered slots never precede the sub-tile: a committed key keeps its
  // position, and the ancestor shown at position n + j is a block row of
  // index >= j, i.e. slot >= n + j.  So when the block ends inside the staged
  // split (the usual case) every gathered slot is staged: gather from LDS;
  // else from the KV pool.  Uniform over the workgroup.
  const bool from_lds = nkeys <= base0 + 64 * nsub;
  // pages of the slots a gather sub-tile can touch, [base0 + 64 g0, n + T):
  // at most four 64-slot pages, fetched once
  const int pw0 = (base0 >> 6) + g0;
  int pgt[4];
  {
    const auto pr = make_rsrc(ptable, (unsigned)(a.ptable_len * 4));
    const unsigned o4 = (unsigned)(pw0 * 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) pgt[i] = (int)__builtin_amdgcn_raw_buffer_load_b32(pr, o4 + 4 * i, 0, 0);
  }
  // row tr's path (lane j holds the block row at depth j + 1) and position;
  // the next row's are fetched while the current one is computed
  const auto pathr = make_rsrc(path, (unsigned)(a.T * 64));
  const auto posr = make_rsrc(pos, (unsigned)(a.T * 4));
  int tr = t_lo + kk;
  uint32_t pth = __builtin_amdgcn_raw_buffer_load_b8(pathr, (unsigned)(tr * 64 + lane), 0, 0);
  int ptr = (int)__builtin_amdgcn_raw_buffer_load_b32(posr, (unsigned)(tr * 4), 0, 0);
  for (; tr <= t_hi; tr += nw) {
    const int dep = __builtin_amdgcn_readfirstlane(ptr) - n;
    const int pth_tr = (int)pth;
    if (tr + nw <= t_hi) {
      pth = __builtin_amdgcn_raw_buffer_load_b8(pathr, (unsigned)((tr + nw) * 64 + lane), 0, 0);
      ptr = (int)__builtin_amdgcn_raw_buffer_load_b32(posr, (unsigned)((tr + nw) * 4), 0, 0);
    }
    // physical slot holding position kp on row tr's path (-1: hidden); the
    // lane shuffle runs on every lane
    auto slot_of = [&](int kp) {
      const int j = min(max(kp - n - 1, 0), 63);
      const int anc = n + (__shfl(pth_tr, j) & 0xff);
      return kp <= n ? kp : (kp - n <= dep ? anc : -1);
    };
    // every column accumulates; only row tr's columns get non-zero weights
    const bool own = colok && t == tr;
    constexpr int NVK = DT == DT_BF16 ? 8 : 4;   // value keys of one PV step per lane
    // value key i of PV step j: bf16 32j + 16(i/4) + 4grp + i%4, fp32 16j + 4grp + i
    auto vkey = [&](int j, int i) {
      return DT == DT_BF16 ? 32 * j + 16 * (i >> 2) + 4 * grp + (i & 3) : 16 * j + 4 * grp + i;
    };
    {
      const int gbase = base0 + 64 * (g0 + gi);
      float mt, lt;
      if (from_lds) {
        // staged row of each key; hidden keys (weight 0) read a staged row
        auto row_of = [&](int kp) {
          const int ps = slot_of(kp);
          return (ps < 0 ? max(n, base0) : ps) - base0;
        };
        int krow[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) krow[kt] = row_of(gbase + 16 * kt + c);
        auto kfn = [&](int kt, int s) {
          const int r = krow[kt];
          return *reinterpret_cast<const uint4*>(Kall + (r >> 6) * LY::KSUB + (r & 63) * KROW +
                                                 (s * KS + grp * EPL) * ESZ);
        };
        int vrow[NVK];
        auto vprep = [&](int j) {
#pragma unroll
          for (int i = 0; i < NVK; ++i) vrow[i] = row_of(gbase + vkey(j, i));
        };
        auto vfn = [&](int dt, int j) {
          const unsigned char* vd = Vall + (16 * dt + c) * VROW;
          auto elt = [&](int i) -> uint32_t {
            const int r = vrow[i];
            const unsigned char* src = vd + (r >> 6) * LY::VSUB + (DT == DT_BF16 ? vt_pos(r & 63) : (r & 63)) * ESZ;
            return DT == DT_BF16 ? (uint32_t)*reinterpret_cast<const uint16_t*>(src)
                                 : *reinterpret_cast<const uint32_t*>(src);
          };
          uint32_t w[4];
          if (DT == DT_BF16) {
#pragma unroll
            for (int h = 0; h < 4; ++h) w[h] = elt(2 * h) | (elt(2 * h + 1) << 16);
          } else {
#pragma unroll
            for (int h = 0; h < 4; ++h) w[h] = elt(h);
          }
          return make_uint4(w[0], w[1], w[2], w[3]);
        };
        subtile_state<DT, HD, false>(qf, kfn, vfn, vprep, gbase, mypos, a.scale_log2, grp, own, mt, lt, o);
      } else {
        // byte offset in the KV pool of slot ps's K row (kv = 0) or V^T column (kv = 1)
        auto off_of = [&](int ps, int kv) {
          if (ps < 0) return OOB;
          const int pi = (ps >> 6) - pw0;             // 0..3 (see pw0)
          const int page = pi == 0 ? pgt[0] : pi == 1 ? pgt[1] : pi == 2 ? pgt[2] : pgt[3];
          return (unsigned)(((((size_t)page * 2 + kv) * a.Hkv + gkv) * 64 * HD) * ESZ +
                            (size_t)(ps & 63) * (kv ? 1 : HD) * ESZ);
        };
        unsigned koff[4];
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) koff[kt] = off_of(slot_of(gbase + 16 * kt + c), 0);
        auto kfn = [&](int kt, int s) {
          return bload<0>(rs, koff[kt] == OOB ? OOB : koff[kt] + (unsigned)((s * KS + grp * EPL) * ESZ));
        };
        unsigned voff[NVK];
        auto vprep = [&](int j) {
#pragma unroll
          for (int i = 0; i < NVK; ++i) voff[i] = off_of(slot_of(gbase + vkey(j, i)), 1);
        };
        auto vfn = [&](int dt, int j) {
          const unsigned drow = (unsigned)((16 * dt + c) * 64 * ESZ);
          auto elt = [&](int i) -> uint32_t {
            const unsigned off = voff[i] == OOB ? OOB : voff[i] + drow;
            return DT == DT_BF16 ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0)
                                 : __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
          };
          uint32_t w[4];
          if (DT == DT_BF16) {
#pragma unroll
            for (int h = 0; h < 4; ++h) w[h] = (elt(2 * h) & 0xffffu) | (elt(2 * h + 1) << 16);
          } else {
#pragma unroll
            for (int h = 0; h < 4; ++h) w[h] = elt(h);
          }
          return make_uint4(w[0], w[1], w[2], w[3]);
        };
        // all value fragments of a PV step are fetched before its MFMAs
        subtile_state<DT, HD, false>(qf, kfn, vfn, vprep, gbase, mypos, a.scale_log2, grp, own, mt, lt, o);
      }
      if (own) {
        m = mt;
        l = lt;
      }
    }
  }
  }

  // sub-tile states -> LDS (over the staged keys, no longer needed); merge in
  // sub-tile order: M = max m, w = 2^(m - M), L = sum l w, O = sum o w.  A
  // gather sub-tile's slot is filled row by row by the waves that computed
  // the rows.
  __syncthreads();
  // state rows [column][HD + 4] floats: a lane's four dims 16dt + 4grp .. +3
  // are one 16-byte chunk (rows padded by 16 bytes: conflict-free)
  constexpr int SROW = HD + 4;
  float* stO = reinterpret_cast<float*>(lds);                          // [ATT_QT][NSUB][16][SROW]
  float* stM = stO + ATT_QT * NSUB * 16 * SROW;                         // [ATT_QT][NSUB][16]
  float* stL = stM + ATT_QT * NSUB * 16;
  auto put_state = [&](int slot, const f32x4 (&ov)[ND], float mv, float lv) {
  float* so = stO + ((size_t)(qi * NSUB + slot) * 16 + c) * SROW;
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) *reinterpret_cast<f32x4*>(so + 16 * dt + 4 * grp) = ov[dt];
  if (grp == 0) {
    stM[(qi * NSUB + slot) * 16 + c] = mv;
    stL[(qi * NSUB + slot) * 16 + c] = lv;
  }
  };
  if (!worker) {
  put_state(st, o, m, l);
  } else {
  if (st > g1) {
    f32x4 z[ND];
#pragma unroll
    for (int i = 0; i < ND; ++i) z[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    put_state(st, z, -INFINITY, 0.f);
  }
  if (qt < nqt && colok && t >= t_lo + kk && (t - t_lo - kk) % nw == 0) put_state(g0 + gi, o, m, l);
  }
  __syncthreads();
  // thread -> (query tile, column, HD/16 dims)
  constexpr int DPT = HD / 16;
  const int mq = threadIdx.x / 256, rest = threadIdx.x % 256;
  const int col = rest & 15, d0 = (rest >> 4) * DPT;
  const int qcol = (qgrp * ATT_QT + mq) * 16 + col;
  if (qcol >= a.ncols) return;
  float M = -INFINITY;
#pragma unroll
  for (int j = 0; j < NSUB; ++j)
  if (stL[(mq * NSUB + j) * 16 + col] > 0.f) M = fmaxf(M, stM[(mq * NSUB + j) * 16 + col]);
  float L = 0.f, O[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) O[e] = 0.f;
#pragma unroll
  for (int j = 0; j < NSUB; ++j) {
  const float lj = stL[(mq * NSUB + j) * 16 + col];
  if (!(lj > 0.f)) continue;
  const float w = exp2f(stM[(mq * NSUB + j) * 16 + col] - M);
  L = fmaf(lj, w, L);
  const float* so = stO + ((size_t)(mq * NSUB + j) * 16 + col) * SROW + d0;
  float sv[DPT];
#pragma unroll
  for (int e = 0; e < DPT; e += 4) *reinterpret_cast<f32x4*>(sv + e) = *reinterpret_cast<const f32x4*>(so + e);
#pragma unroll
  for (int e = 0; e < DPT; ++e) O[e] = fmaf(sv[e], w, O[e]);
  }
  float* out = a.part + (((size_t)sp * a.Hkv + gkv) * ((size_t)a.B * a.ncols) + (size_t)b * a.ncols + qcol) * (HD + 2);
#pragma unroll
  for (int e = 0; e < DPT; e += 4)
  *reinterpret_cast<float4*>(out + d0 + e) = make_float4(O[e], O[e + 1], O[e + 2], O[e + 3]);
  if (d0 == 0) {
  out[HD] = M;
  out[HD + 1] = L;
  }
}

template <int DT, int HD, bool TREE>
__global__ __launch_bounds__(att_threads(TREE)) void attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[AttnLds<DT, HD, att_threads(TREE)>::BYTES];
  attn_block<DT, HD, TREE>(a, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

// Split attention for blocks with many query tiles (long drafts, batches of
// sequences).  Workgroup (KV head g, split sp, sequence b, group qg of nqg)
// stages the split once and its 8 waves walk the sequence's query tiles qg*8 +
// wave, + 8 nqg, ...; a wave computes all four sub-tiles of a query tile
// itself: the scores of every sub-tile first (their maxima give the split
// maximum M), then each sub-tile's weights and value products, folded in
// sub-tile order with weight 2^(m_j - M).  Every operation on a column's
// values is the one attn_kernel performs (same sub-tile arithmetic, same merge
// order), so the two kernels give bitwise equal states; this one only avoids
// staging the split again for every four query tiles.
constexpr int WIDE_THREADS = 512;
constexpr int WIDE_MIN_QT = 13;   // query tiles per sequence from which the wide kernel is used

// (the body of one workgroup, block (bx, by, bz) of the grid, with its LDS at
// lds: AttnLds<DT, HD, WIDE_THREADS>::KV_BYTES)
template <int DT, int HD>
__device__ __forceinline__ void attn_wide_block(AttnArgs a, int nqg, int bx, int by, int bz, unsigned char* lds) {
  using LY = AttnLds<DT, HD, WIDE_THREADS>;
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL, ESZ = Geo<DT>::ESZ;
  constexpr int NS = HD / KS, ND = HD / 16;
  constexpr int ROWB = LY::ROWB, KROW = LY::KROW, VROW = LY::VROW;
  const unsigned char* Kall = lds;
  const unsigned char* Vall = lds + NSUB * LY::KSUB;

  const int nqt = (a.ncols + 15) / 16;
  const int gkv = bx, sp = by, b = bz / nqg, qg = bz % nqg;
  const int rb = b * a.T;
  const int* pos = a.pos + rb;
  const int* ptable = a.ptable + b * a.ptable_len;
  const uint2 inf = bload64<0>(make_rsrc(a.info + 4 * b, 8), 0);
  const uint4 p4 = split_pages(a, ptable, sp * SPLIT);   // (same round trip)
  const int n = __builtin_amdgcn_readfirstlane((int)inf.x);
  if (sp >= __builtin_amdgcn_readfirstlane((int)inf.y)) return;   // the grid covers the longest context
  if (a.split_mode == 1 && sp >= (n + 1) / SPLIT) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int grp = lane >> 4, c = lane & 15;
  const int nkeys = n + a.T;
  const int base0 = sp * SPLIT;
  const int nsub = min(NSUB, (nkeys - base0 + 63) / 64);
  stage_split<DT, HD, WIDE_THREADS>(a, p4, gkv, base0, nsub, nkeys, lds);
  __syncthreads();

  const auto qr = make_rsrc(a.q, (unsigned)((size_t)a.B * a.T * a.H * ROWB));
  for (int qt = qg * 8 + wv; qt < nqt; qt += nqg * 8) {   // uniform per wave
    const int qc = qt * 16 + c;
    const bool colok = qc < a.ncols;
    const int t = colok ? qc / a.G : 0;
    const int head = gkv * a.G + (colok ? qc % a.G : 0);
    const int mypos = colok ? pos[t] : -1;
    uint4 qf[NS];
    const unsigned qb = (unsigned)(((size_t)(rb + t) * a.H + head) * ROWB);
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = bload<0>(qr, colok ? qb + (unsigned)((s * KS + grp * EPL) * ESZ) : OOB);
    f32x4 sc[NSUB][4];
    float mj[NSUB];
    float M = -INFINITY;
#pragma unroll
    for (int st = 0; st < NSUB; ++st) {
      mj[st] = -INFINITY;
      if (st < nsub) {
        const unsigned char* Ks = Kall + st * LY::KSUB;
        auto kfn = [&](int kt, int s) {
          return *reinterpret_cast<const uint4*>(Ks + (size_t)(16 * kt + c) * KROW + (s * KS + grp * EPL) * ESZ);
        };
        subtile_scores<DT, HD>(qf, kfn, base0 + st * 64, mypos, a.scale_log2, grp, sc[st], mj[st]);
      }
      if (mj[st] > -INFINITY && mj[st] < INFINITY) M = fmaxf(M, mj[st]);
    }
    float L = 0.f;
    f32x4 O[ND];
#pragma unroll
    for (int i = 0; i < ND; ++i) O[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < NSUB; ++st) {
      if (st >= nsub) continue;
      const unsigned char* Vt = Vall + st * LY::VSUB;
      auto vfn = [&](int dt, int j) {
        const unsigned char* vr = Vt + (size_t)(16 * dt + c) * VROW;
        if (DT == DT_BF16) return *reinterpret_cast<const uint4*>(vr + (32 * j + 8 * grp) * ESZ);   // (vt_pos)
        return *reinterpret_cast<const uint4*>(vr + (16 * j + 4 * grp) * ESZ);
      };
      f32x4 oj[ND];
#pragma unroll
      for (int i = 0; i < ND; ++i) oj[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      float lj;
      subtile_values<DT, HD, false>(sc[st], mj[st], vfn, [](int) {}, grp, true, lj, oj);
      if (lj > 0.f) {
        const float w = exp2f(mj[st] - M);
        L = fmaf(lj, w, L);
#pragma unroll
        for (int dt = 0; dt < ND; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) O[dt][r] = fmaf(oj[dt][r], w, O[dt][r]);
      }
    }
    if (colok) {
      float* out = a.part + (((size_t)sp * a.Hkv + gkv) * ((size_t)a.B * a.ncols) + (size_t)b * a.ncols + qc) * (HD + 2);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
        *reinterpret_cast<float4*>(out + 16 * dt + 4 * grp) = make_float4(O[dt][0], O[dt][1], O[dt][2], O[dt][3]);
      if (grp == 0) {
        out[HD] = M;
        out[HD + 1] = L;
      }
    }
  }
}

template <int DT, int HD>
__global__ __launch_bounds__(WIDE_THREADS) void attn_wide_kernel(AttnArgs a, int nqg) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[AttnLds<DT, HD, WIDE_THREADS>::KV_BYTES];
  attn_wide_block<DT, HD>(a, nqg, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

// A large tree's attention in one launch: first the workgroups of
// attn_kernel<TREE> over the splits holding the tree's rows (tail: grid
// Hkv x ty x tz; the longest), then those of attn_wide_kernel over the splits
// below them (lin: grid Hkv x wy x wz), so the two sets run side by side
// instead of one after the other.  Every workgroup runs exactly the arithmetic
// of its own kernel.
template <int DT, int HD>
__global__ __launch_bounds__(WIDE_THREADS) void attn_tree_wide_kernel(AttnArgs tail, AttnArgs lin, int nqg,
                                                                     int ty, int tz, int wy) {
  static_assert(att_threads(true) == WIDE_THREADS, "one workgroup size for both parts");
  constexpr int B1 = AttnLds<DT, HD, WIDE_THREADS>::BYTES, B2 = AttnLds<DT, HD, WIDE_THREADS>::KV_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[B1 > B2 ? B1 : B2];
  const int hk = tail.Hkv, ntree = hk * ty * tz;
  const int id = blockIdx.x;
  if (id < ntree) {
    attn_block<DT, HD, true>(tail, id % hk, id / hk % ty, id / (hk * ty), lds);
  } else {
    const int w = id - ntree;
    attn_wide_block<DT, HD>(lin, nqg, w % hk, w / hk % wy, w / (hk * wy), lds);
  }
}

constexpr int MAX_SPLITS = 32;   // committed + block positions <= 8192

// Merge the splits of every (row, head) in split order; write the attention
// output as packed activations of the O projection.  4 dims per thread.  The
// state of every split of the attention grid (max_splits, fixed at launch) is
// fetched in one batch; only the first info[1] of the row's sequence take part.
constexpr int CMB_THREADS = 128;   // 4 (row, head) columns per workgroup at head_dim 128

template <int DT, int HD>
__global__ __launch_bounds__(CMB_THREADS) void attn_combine_kernel(const float* __restrict__ part,
                                                              const int* __restrict__ info, int max_splits,
                                                              int Hkv, int G, int ncols, int H, int T,
                                                              void* __restrict__ xout, int x_S) {
  // ncols: query columns of the whole block (all sequences); row t belongs to
  // sequence t / T
  // CMB_THREADS * 4 / HD (row, head) columns per workgroup, HD / 4 threads of 4 dims each
  constexpr int TPC = HD / 4;
  const int pq = blockIdx.x * (CMB_THREADS / TPC) + threadIdx.x / TPC;
  if (pq >= ncols / G * H) return;
  const int t = pq / H, j = pq % H;
  const int gkv = j / G, qc = t * G + (j % G);
  const int dim = (threadIdx.x % TPC) * 4;
  float ms[MAX_SPLITS], ls[MAX_SPLITS];
  float4 os[MAX_SPLITS];
  // vector (buffer) loads throughout: the (m, l) addresses are uniform, and
  // scalar loads of them would be serialised one round trip at a time
  const auto pr = make_rsrc(part, (unsigned)((size_t)max_splits * Hkv * ncols * (HD + 2) * 4));
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s) {
    if (s < max_splits) {
      const unsigned off = (unsigned)((((size_t)s * Hkv + gkv) * ncols + qc) * (HD + 2) * 4);
      const uint2 ml = bload64<0>(pr, off + HD * 4);
      ms[s] = __uint_as_float(ml.x);
      ls[s] = __uint_as_float(ml.y);
      const uint4 ov = bload<0>(pr, off + (unsigned)dim * 4);
      os[s] = make_float4(__uint_as_float(ov.x), __uint_as_float(ov.y), __uint_as_float(ov.z), __uint_as_float(ov.w));
    }
  }
  const int nsplit = info[4 * (t / T) + 1];
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s)
    if (s < nsplit && ls[s] > 0.f) M = fmaxf(M, ms[s]);
  float L = 0.f, O[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s) {
    if (s >= nsplit || !(ls[s] > 0.f)) continue;
    const float w = exp2f(ms[s] - M);
    L = fmaf(ls[s], w, L);
    O[0] = fmaf(os[s].x, w, O[0]);
    O[1] = fmaf(os[s].y, w, O[1]);
    O[2] = fmaf(os[s].z, w, O[2]);
    O[3] = fmaf(os[s].w, w, O[3]);
  }
  const size_t fi = frag_index<DT>(t, j * HD + dim, x_S);
  if (DT == DT_BF16) {
    const uint2 u = make_uint2(f2bf_bits(O[0] / L) | (f2bf_bits(O[1] / L) << 16),
                               f2bf_bits(O[2] / L) | (f2bf_bits(O[3] / L) << 16));
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(xout) + fi) = u;
  } else {
    *reinterpret_cast<float4*>(reinterpret_cast<float*>(xout) + fi) =
        make_float4(O[0] / L, O[1] / L, O[2] / L, O[3] / L);
  }
}

// ------------------------------------------------------- argmax and accept --

__global__ __launch_bounds__(256) void argmax_kernel(const unsigned long long* __restrict__ amax,
                                                     int n_tiles, int* __restrict__ greedy) {
  __shared__ unsigned long long sh[256];
  const int t = blockIdx.x;
  unsigned long long best = 0;
  for (int i = threadIdx.x; i < n_tiles; i += 256) {
    const unsigned long long k = amax[(size_t)t * n_tiles + i];
    best = k > best ? k : best;
  }
  sh[threadIdx.x] = best;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      const unsigned long long o = sh[threadIdx.x + w];
      if (o > sh[threadIdx.x]) sh[threadIdx.x] = o;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) greedy[t] = (int)(0xffffffffu - (uint32_t)(sh[0] & 0xffffffffull));
}

// Value of an ordered key (inverse of amax_key; -0 comes back as +0).
__device__ __forceinline__ float key_value(unsigned long long key) {
  const uint32_t ord = (uint32_t)(key >> 32);
  return __uint_as_float((ord & 0x80000000u) ? (ord & 0x7fffffffu) : ~ord);
}
__device__ __forceinline__ int key_index(unsigned long long key) {
  return (int)(0xffffffffu - (uint32_t)(key & 0xffffffffull));
}

// Entropy-aware top-k verification of row t (Eq. 9-10), one wave per row.
// The row's top-k tokens (k = info[4b+2] <= 8, ties ranked by lower id) come
// from merging the per-chunk top-8 keys; their probabilities renormalised
// over the k tokens give the normalised entropy H = -sum q log q / log k, in
// float64, and the threshold tau = max(1, ceil(k H)) (dynamic, info[4b+3] != 0)
// or tau = k (fixed).  The draft token of row t + 1 is accepted when it is one
// of the first tau tokens.  verdict[t] = tau | accepted << 8; greedy[t] is the
// top-1 token, i.e. the greedy token of the row.
__global__ __launch_bounds__(64) void topk_select_kernel(const unsigned long long* __restrict__ cand, int nchunk,
                                                         const int* __restrict__ tok,
                                                         const int* __restrict__ info, int T,
                                                         int* __restrict__ greedy, int* __restrict__ verdict) {
  const int t = blockIdx.x, lane = threadIdx.x;
  const int b = t / T, tt = t - b * T;
  unsigned long long k8[8] = {0ull, 0ull, 0ull, 0ull, 0ull, 0ull, 0ull, 0ull}, top[8];
  const unsigned long long* row = cand + (size_t)t * nchunk * 8;
  for (int i = lane; i < nchunk * 8; i += 64) {
    const unsigned long long x = row[i];
    if (x > k8[7]) {
      k8[7] = x;
#pragma unroll
      for (int j = 7; j > 0; --j) cx_desc(k8[j - 1], k8[j]);
    }
  }
  wave_top8(k8, top);
  const int kk = info[4 * b + 2], dyn = info[4 * b + 3];
  int tau = kk;
  if (kk > 1) {
    const double v0 = (double)key_value(top[0]);
    double e[8], S = 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      e[j] = (j < kk && top[j] != 0ull) ? exp((double)key_value(top[j]) - v0) : 0.0;
      S += e[j];
    }
    double hs = 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const double q = e[j] / S;
      if (q > 0.0) hs += q * log(q);
    }
    const double H = -hs / log((double)kk);
    if (dyn) {
      const double up = ceil((double)kk * H);
      tau = up < 1.0 ? 1 : (up > (double)kk ? kk : (int)up);
    }
  } else {
    tau = 1;
  }
  int hit = 0;
  if (tt + 1 < T) {
    const int d = tok[t + 1];
#pragma unroll
    for (int j = 0; j < 8; ++j) hit |= (j < tau && top[j] != 0ull && key_index(top[j]) == d) ? 1 : 0;
  }
  if (lane == 0) {
    greedy[t] = key_index(top[0]);
    verdict[t] = tau | (hit << 8);
  }
}

// Stochastic verification (Eq. 4), step 1, one workgroup per row: the row's
// maximum logit M (from the chunk maxima), e_v = exp((l_v - M) / temp) (kept
// in ebuf[t] for the draw that may follow at this row) and S = sum_v e_v, in
// float64 with a fixed summation order; draft row t (t + 1 < T) accepts token
// d = tok[t + 1] when eps_t * q_t[d] < p_t[d] = e_d / S, with q_t[d] from the
// draft distribution (1 when none is given: a greedy draft).  verdict[t] bit
// 8 = accepted; greedy[t] = the row's argmax; rowstat[t] = (M, S).
struct SampleParams {
  unsigned long long q;   // device address of the draft distribution [K][V] fp32, or 0
  float temperature;
  int residual;
};
constexpr int SAMPLE_MAX_GROUPS = 4096;   // 64-token groups: vocabularies up to 262144 tokens

__device__ __forceinline__ double sample_weight(const double* e, const float* q, int d, int v, double S, bool resid) {
  if (!resid) return e[v];
  const double p = e[v] / S;
  const double qv = q ? (double)q[v] : (v == d ? 1.0 : 0.0);
  return p > qv ? p - qv : 0.0;
}

__global__ __launch_bounds__(256) void sample_stats_kernel(const float* __restrict__ logits,
                                                           const unsigned long long* __restrict__ amax, int nchunk,
                                                           int V, const int* __restrict__ tok, int T,
                                                           const float* __restrict__ eps,
                                                           const unsigned char* __restrict__ sparam,
                                                           double* __restrict__ rowstat, double* __restrict__ ebuf,
                                                           int* __restrict__ greedy, int* __restrict__ verdict) {
  __shared__ double sh[256];
  __shared__ unsigned long long shk[256];
  const int t = blockIdx.x, tid = threadIdx.x;
  const SampleParams sp = *reinterpret_cast<const SampleParams*>(sparam);
  unsigned long long best = 0;
  for (int i = tid; i < nchunk; i += 256) best = amax[(size_t)t * nchunk + i] > best ? amax[(size_t)t * nchunk + i] : best;
  shk[tid] = best;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w && shk[tid + w] > shk[tid]) shk[tid] = shk[tid + w];
    __syncthreads();
  }
  const unsigned long long key = shk[0];
  const double M = (double)key_value(key), it = 1.0 / (double)sp.temperature;
  const float* row = logits + (size_t)t * V;
  double* e = ebuf + (size_t)t * V;
  double acc = 0.0;
  for (int v = tid; v < V; v += 256) {
    const double ev = exp(((double)row[v] - M) * it);
    e[v] = ev;
    acc += ev;
  }
  sh[tid] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) sh[tid] += sh[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    const double S = sh[0];
    rowstat[2 * t] = M;
    rowstat[2 * t + 1] = S;
    greedy[t] = key_index(key);
    int ok = 0;
    if (t + 1 < T) {
      const int d = tok[t + 1];
      const double pd = exp(((double)row[d] - M) * it) / S;
      const double qd = sp.q ? (double)reinterpret_cast<const float*>(sp.q)[(size_t)t * V + d] : 1.0;
      ok = (double)eps[t] * qd < pd ? 1 : 0;
    }
    verdict[t] = ok << 8;
  }
}

// Stochastic verification, step 2 (after the acceptance scan), one workgroup:
// row a = result[0] draws the next token by inverse CDF with u = unif[a] over
// w_v = max(0, p_v - q_v) (a rejected draft row with `residual`; p instead
// when the residual vanishes) or over e_v, proportional to p (the bonus row,
// or no residual): the smallest v whose cumulative weight in token order
// exceeds u times the total.  The vocabulary is cut into 64-token groups;
// group sums (tiles of 64 groups transposed through LDS, each summed in token
// order), runs of groups per thread, run offsets in thread order, then an
// inclusive scan over the chosen group's tokens.  float64; rounding that
// leaves the target past every sum picks the last token of non-zero weight.
__global__ __launch_bounds__(256) void resample_kernel(const double* __restrict__ ebuf, int V, const int* __restrict__ tok,
                                                       int T, const float* __restrict__ unif,
                                                       const unsigned char* __restrict__ sparam,
                                                       const double* __restrict__ rowstat, int* __restrict__ result) {
  __shared__ double tile[64][65];
  __shared__ double gs[SAMPLE_MAX_GROUPS];
  __shared__ double run_s[256], run_o[257];
  __shared__ int sel[2];
  __shared__ double sel_off;
  const int tid = threadIdx.x, lane = tid & 63;
  const SampleParams sp = *reinterpret_cast<const SampleParams*>(sparam);
  const int a = result[0];
  const int K = T - 1;
  const double S = rowstat[2 * a + 1];
  const double* e = ebuf + (size_t)a * V;
  const bool draft_row = a < K;
  const int d = draft_row ? tok[a + 1] : -1;
  const float* q = (draft_row && sp.q) ? reinterpret_cast<const float*>(sp.q) + (size_t)a * V : nullptr;
  bool resid = draft_row && sp.residual;
  const int ng = (V + 63) / 64, per = (ng + 255) / 256;
  const int r0 = min(ng, tid * per), r1 = min(ng, r0 + per);
  for (int pass = 0; pass < 2; ++pass) {
    for (int base = 0; base < ng; base += 64) {
      for (int k = tid; k < 64 * 64; k += 256) {
        const int v = base * 64 + k;
        tile[k >> 6][k & 63] = v < V ? sample_weight(e, q, d, v, S, resid) : 0.0;
      }
      __syncthreads();
      if (tid < 64 && base + tid < ng) {
        double sum = 0.0;
        for (int j = 0; j < 64; ++j) sum += tile[tid][j];
        gs[base + tid] = sum;
      }
      __syncthreads();
    }
    double run = 0.0;
    for (int g = r0; g < r1; ++g) run += gs[g];
    run_s[tid] = run;
    __syncthreads();
    if (tid == 0) {
      double o = 0.0;
      for (int i = 0; i < 256; ++i) {
        run_o[i] = o;
        o += run_s[i];
      }
      run_o[256] = o;
    }
    __syncthreads();
    if (!(resid && !(run_o[256] > 0.0))) break;
    resid = false;   // p == q: nothing to correct, draw from p
    __syncthreads();
  }
  const double target = (double)unif[a] * run_o[256];
  if (tid == 0) {
    sel[0] = -1;
    sel[1] = -1;
  }
  __syncthreads();
  // the run, then the group, holding the target; else the last group of non-zero weight
  if (r0 < r1 && target >= run_o[tid] && target < run_o[tid] + run_s[tid]) {
    double c = run_o[tid];
    for (int g = r0; g < r1; ++g) {
      if (gs[g] > 0.0 && target < c + gs[g]) {
        sel[0] = g;
        sel_off = c;
        break;
      }
      c += gs[g];
    }
  }
  __syncthreads();
  if (tid == 0 && sel[0] < 0) {
    double c = 0.0;
    for (int g = 0; g < ng; ++g) {
      if (gs[g] > 0.0) {
        sel[0] = g;
        sel_off = c;
      }
      c += gs[g];
    }
    if (sel[0] < 0) sel[0] = 0;
  }
  __syncthreads();
  if (tid < 64) {
    const int g = sel[0];
    const int v = g * 64 + lane;
    const double wv = v < V ? sample_weight(e, q, d, v, S, resid) : 0.0;
    double incl = wv;   // inclusive scan over the group in token order
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const double y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    const unsigned long long over = __ballot(wv > 0.0 && sel_off + incl > target);
    const unsigned long long pos = __ballot(wv > 0.0);
    int chosen;
    if (over) chosen = g * 64 + (__ffsll((long long)over) - 1);
    else chosen = pos ? g * 64 + (63 - __clzll((long long)pos)) : g * 64;
    if (lane == 0) result[1] = chosen;
  }
}

// result[0] = accepted rows a, result[1] = next token, result[2..2+a) = accepted
// block rows in depth order (mode 3: result[2..2+K) = the threshold tau of
// every draft row).  Mode 0 (prefill) commits every row.
__global__ __launch_bounds__(64) void accept_kernel(const int* __restrict__ tok,
                                                    const int* __restrict__ prow,
                                                    const int* __restrict__ greedy,
                                                    const int* __restrict__ verdict, int T, int mode,
                                                    int* __restrict__ result, int rec) {
  // workgroup b: sequence b, rows b*T .. b*T + T - 1, result record b (rec ints)
  tok += blockIdx.x * T;
  prow += blockIdx.x * T;
  greedy += blockIdx.x * T;
  verdict += blockIdx.x * T;
  result += blockIdx.x * rec;
  const int lane = threadIdx.x;
  const int K = T - 1;
  if (mode == 0) {
    if (lane == 0) {
      result[0] = T - 1;
      result[1] = greedy[T - 1];
    }
    return;
  }
  if (mode == 1 || mode == 3 || mode == 4) {
    // draft d_{i+1} (row i+1) is checked against row i: its greedy token
    // (mode 1) or its verdict (mode 3: top-k, mode 4: stochastic); the first
    // failing row, found 64 rows at a time, is a.  Mode 3 also records every
    // row's threshold.
    int a = K;
    for (int i0 = 0; i0 < K; i0 += 64) {
      const int i = i0 + lane;
      bool fails = false;
      if (i < K) {
        if (mode == 1) {
          fails = tok[i + 1] != greedy[i];
        } else if (mode == 4) {
          fails = !((verdict[i] >> 8) & 1);
        } else {
          const int vd = verdict[i];
          fails = !((vd >> 8) & 1);
          result[2 + i] = vd & 0xff;
        }
      }
      const unsigned long long b = __ballot(fails);
      if (b && a == K) a = i0 + __ffsll((long long)b) - 1;
      if (mode != 3 && a != K) break;
    }
    if (lane == 0) {
      result[0] = a;
      result[1] = greedy[a];
    }
    if (mode != 3)
      for (int i = lane; i < a; i += 64) result[2 + i] = i + 1;
    return;
  }
  // tree walk from row 0 (trees have at most 64 nodes)
  int cur = 0, a = 0;
  for (;;) {
    const bool hit = lane < K && prow[lane + 1] == cur && tok[lane + 1] == greedy[cur];
    const unsigned long long b = __ballot(hit);
    if (!b) break;
    const int row = __ffsll((long long)b);   // lowest node index i -> row i + 1
    if (lane == 0) result[2 + a] = row;
    cur = row;
    ++a;
  }
  if (lane == 0) {
    result[0] = a;
    result[1] = greedy[cur];
  }
}

// Move K/V of accepted tree rows to consecutive slots n+1.. in depth order.
template <int DT, int HD>
__global__ __launch_bounds__(256) void compact_kernel(void* __restrict__ kv_pool, size_t layer_stride,
                                                      const int* __restrict__ ptable,
                                                      const int* __restrict__ result,
                                                      const int* __restrict__ info, int Hkv,
                                                      int ptable_len, int rec) {
  constexpr int ESZ = Geo<DT>::ESZ;
  // blockIdx.y: sequence
  ptable += blockIdx.y * ptable_len;
  result += blockIdx.y * rec;
  const int n = info[4 * blockIdx.y];
  const int layer = blockIdx.x / Hkv, g = blockIdx.x % Hkv;
  const int a = result[0];
  unsigned char* lb = reinterpret_cast<unsigned char*>(kv_pool) + layer * layer_stride * ESZ;
  const size_t hs = (size_t)64 * HD;
  // pass 1: read all sources; pass 2: write all destinations (sources never
  // lie below their destinations, but a source may be another's destination)
  __shared__ __attribute__((aligned(16))) unsigned char kbuf[64 * HD * ESZ];
  __shared__ __attribute__((aligned(16))) unsigned char vbuf[64 * HD * ESZ];
  for (int i = threadIdx.x; i < a * HD; i += 256) {
    const int r = i / HD, dim = i % HD;
    const int src = n + result[2 + r];
    const int page = ptable[src >> 6], sp = src & 63;
    const unsigned char* kb = lb + ((((size_t)page * 2 + 0) * Hkv + g) * hs) * ESZ;
    const unsigned char* vb = lb + ((((size_t)page * 2 + 1) * Hkv + g) * hs) * ESZ;
    for (int e = 0; e < ESZ; ++e) {
      kbuf[(r * HD + dim) * ESZ + e] = kb[((size_t)sp * HD + dim) * ESZ + e];
      vbuf[(r * HD + dim) * ESZ + e] = vb[((size_t)dim * 64 + sp) * ESZ + e];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < a * HD; i += 256) {
    const int r = i / HD, dim = i % HD;
    const int dst = n + 1 + r;
    const int page = ptable[dst >> 6], sp = dst & 63;
    unsigned char* kb = lb + ((((size_t)page * 2 + 0) * Hkv + g) * hs) * ESZ;
    unsigned char* vb = lb + ((((size_t)page * 2 + 1) * Hkv + g) * hs) * ESZ;
    for (int e = 0; e < ESZ; ++e) {
      kb[((size_t)sp * HD + dim) * ESZ + e] = kbuf[(r * HD + dim) * ESZ + e];
      vb[((size_t)dim * 64 + sp) * ESZ + e] = vbuf[(r * HD + dim) * ESZ + e];
    }
  }
}

// ------------------------------------------------------------- step driver --

// Runs `launch` bracketed by profiling events when class `c` is selected.  A
// block with more timed launches than event pairs fails (it is never timed
// in part).
template <typename F>
static hipError_t timed(Prof* prof, int c, hipStream_t st, F&& launch) {
  const bool on = prof && prof->on(c);
  if (on && prof->used >= prof->cap) {
    prof->overflow = true;
    return hipErrorInvalidValue;
  }
  hipError_t e;
  if (on && (e = hipEventRecord(prof->ev[2 * prof->used], st)) != hipSuccess) return e;
  if ((e = launch()) != hipSuccess) return e;
  if (on) {
    if ((e = hipEventRecord(prof->ev[2 * prof->used + 1], st)) != hipSuccess) return e;
    prof->cls[prof->used++] = c;
  }
  return hipSuccess;
}

// ------------------------------------------------------ streaming read --
//
// Measurement aid: the HBM read rate a plain streaming kernel reaches on this
// part (the achievable bandwidth the verify step is also compared with).
// One workgroup per CU reads a contiguous chunk of the buffer: its four waves
// take 1 KB segments round-robin, eight non-temporal 16-byte loads in flight
// per thread (the pattern of the GEMMs' weight streams; a grid-stride walk
// over the whole buffer reaches about 15% less).  The loaded words are folded
// into a value that is stored only in a case that does not occur for the data
// measured (so the loads cannot be dropped).
constexpr int STREAM_THREADS = 256, STREAM_UNROLL = 8, STREAM_BLOCKS = 256;

__global__ __launch_bounds__(STREAM_THREADS) void stream_read_kernel(const u32x4* __restrict__ p, size_t n16,
                                                                     unsigned* __restrict__ sink) {
  constexpr int W = STREAM_THREADS / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  // chunk of this workgroup: nseg whole 1 KB segments from base (the last
  // workgroup also reads the segments and 16-byte words left over)
  const size_t seg_all = n16 / 64, per = seg_all / gridDim.x;
  const u32x4* base = p + (size_t)blockIdx.x * per * 64;
  const size_t nseg = blockIdx.x + 1 == gridDim.x ? seg_all - (size_t)blockIdx.x * per : per;
  uint32_t acc = 0;
  size_t s = wv;
  for (; s + (size_t)(STREAM_UNROLL - 1) * W < nseg; s += (size_t)STREAM_UNROLL * W) {
    u32x4 v[STREAM_UNROLL];
#pragma unroll
    for (int j = 0; j < STREAM_UNROLL; ++j) v[j] = __builtin_nontemporal_load(base + (s + (size_t)j * W) * 64 + lane);
    __builtin_amdgcn_sched_barrier(0);   // all eight requested before the first is used
#pragma unroll
    for (int j = 0; j < STREAM_UNROLL; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  for (; s < nseg; s += W) {
    const u32x4 v = __builtin_nontemporal_load(base + s * 64 + lane);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (blockIdx.x + 1 == gridDim.x)   // the words after the last whole segment
    for (size_t i = seg_all * 64 + threadIdx.x; i < n16; i += STREAM_THREADS) {
      const u32x4 v = __builtin_nontemporal_load(p + i);
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

hipError_t run_stream_read(const void* buf, size_t bytes, unsigned* sink, hipStream_t st) {
  const size_t n16 = bytes / 16;
  if (n16 < (size_t)64 * STREAM_BLOCKS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stream_read_kernel, dim3(STREAM_BLOCKS), dim3(STREAM_THREADS), 0, st,
                     reinterpret_cast<const u32x4*>(buf), n16, sink);
  return hipGetLastError();
}

int gemm_slices_for(int K, int dt) { return gemm_slices(K / ks_of(dt)); }

size_t capture_bytes(int L, int d, int qdim, int kvdim, int F, int dt, int R) {
  const size_t esz = esz_of(dt), R16 = (size_t)(R + 15) / 16 * 16;
  const size_t layer = esz * (R16 * (2 * (size_t)d + qdim + F) + (size_t)R * (qdim + 2 * (size_t)kvdim));
  return layer * L + esz * R16 * d;
}

template <int DT, int HD>
static hipError_t forward_t(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  constexpr int KS = Geo<DT>::KS;
  const int T = s.T, B = s.B, R = T * B;   // rows per sequence, sequences, rows
  const int d = m.d, qdim = m.H * m.hd, qkvN = qdim + 2 * m.Hkv * m.hd;
  const int Sd = d / KS, Sq = qdim / KS, Sf = m.F / KS;
  const int sk_d = gemm_slices(Sd), sk_q = gemm_slices(Sq), sk_f = gemm_slices(Sf);
  const size_t layer_elems = (size_t)m.max_pages * 2 * m.Hkv * 64 * m.hd;
  hipError_t e;
  auto last = [] { return hipGetLastError(); };
  // test aid: per layer x_attn | q | k | v | o | x_ffn | z, then x_final
  // (ee_capture); packed buffers of R16 rows
  constexpr size_t ESZ = Geo<DT>::ESZ;
  const size_t R16 = (size_t)(R + 15) / 16 * 16, kvdim = (size_t)m.Hkv * m.hd;
  const size_t c_q = R16 * d * ESZ, c_k = c_q + (size_t)R * qdim * ESZ, c_o = c_k + 2 * (size_t)R * kvdim * ESZ;
  const size_t c_xf = c_o + R16 * qdim * ESZ, c_z = c_xf + R16 * d * ESZ, c_layer = c_z + R16 * m.F * ESZ;
  auto cap = [&](int l, size_t off, const void* src, size_t bytes) {
    return hipMemcpyAsync(s.cap + (size_t)l * c_layer + off, src, bytes, hipMemcpyDeviceToDevice, st);
  };

  if ((e = timed(prof, PC_NORM, st, [&] {
         hipLaunchKernelGGL((resid_kernel<DT, 0>), dim3((d + RES_COLS - 1) / RES_COLS, R), dim3(RES_THREADS), 0, st,
                            m.embed, w.tok, w.h, w.part, 1, R, m.layers[0].attn_gain, d, (void*)w.xbuf, Sd, w.ssq);
         return last();
       })) != hipSuccess)
    return e;
  if (s.cap && (e = cap(0, 0, w.xbuf, R16 * d * ESZ)) != hipSuccess) return e;

  const int G = m.H / m.Hkv, ncols = T * G;   // query columns per sequence
  // the grid covers the splits of the block's longest context; a shorter
  // sequence's splits beyond its own exit at once
  const int nsplit = s.splits;
  if (nsplit < 1 || nsplit > w.max_splits || nsplit > MAX_SPLITS) return hipErrorInvalidValue;
  const int nqt = (ncols + 15) / 16;
  const int pairs = (m.H + 2 * m.Hkv) * (m.hd / 2);
  const bool fused = fused_proj(d, qdim, m.hd, DT);

  for (int l = 0; l < m.L; ++l) {
    const LayerPtrs& lp = m.layers[l];
    void* kvl = reinterpret_cast<unsigned char*>(m.kv_pool) + l * layer_elems * Geo<DT>::ESZ;
    // QKV projection, then rotary + KV append (in the projection's epilogue
    // when fused, else a kernel of their own)
    if (fused) {
      EpArgs qa{};
      qa.w = lp.wqkv; qa.x = w.xbuf; qa.S = Sd; qa.n_tiles = qkvN / 16; qa.n_items = qkvN / 32;
      qa.ssq = w.ssq; qa.d = d; qa.eps = m.eps;
      qa.H = m.H; qa.Hkv = m.Hkv; qa.hd = m.hd; qa.pos = w.pos; qa.rope = m.rope; qa.rowslot = w.slot;
      qa.q = w.q; qa.kv_layer = kvl; qa.kv_cap = s.cap ? (void*)(s.cap + (size_t)l * c_layer + c_k) : nullptr;
      if ((e = timed(prof, PC_QKV, st, [&] { return gemm_ep<DT, EP_ROPE>(qa, R, st); })) != hipSuccess) return e;
    } else {
    if ((e = timed(prof, PC_QKV, st, [&] { return gemm<DT>(lp.wqkv, w.xbuf, qkvN, d, R, w.part, st); })) != hipSuccess)
      return e;
    if ((e = timed(prof, PC_FINISH, st, [&] {
           hipLaunchKernelGGL((qkv_finish_kernel<DT>), dim3((pairs + 255) / 256, R), dim3(256), 0, st, w.part,
                              sk_d, R, qkvN, m.H, m.Hkv, m.hd, w.pos, m.rope, w.slot, w.q, kvl, w.ssq, d, m.eps,
                              s.cap ? (void*)(s.cap + (size_t)l * c_layer + c_k) : nullptr);
           return last();
         })) != hipSuccess)
      return e;
    }
    if (s.cap && (e = cap(l, c_q, w.q, (size_t)R * qdim * ESZ)) != hipSuccess) return e;
    // attention
    AttnArgs aa{};
    aa.q = w.q; aa.kv_layer = kvl; aa.ptable = w.ptable; aa.pos = w.pos; aa.path = w.path;
    aa.info = w.info;
    aa.T = T; aa.H = m.H; aa.Hkv = m.Hkv; aa.G = G; aa.ncols = ncols; aa.B = B;
    aa.tree = s.mode == 2;
    aa.scale_log2 = 1.4426950408889634f / sqrtf((float)m.hd);
    aa.part = w.attn_part;
    aa.max_pages = m.max_pages;
    aa.ptable_len = w.ptable_len;
    if ((e = timed(prof, PC_ATTN, st, [&] {
           // KV head fastest (one head per XCD L2); ATT_QT query tiles per workgroup
           const int qt = att_qt(aa.tree);
           const bool wide = nqt >= WIDE_MIN_QT;
           if (aa.tree && wide) {
             // a large tree: the splits below its rows hold keys every row sees
             // unmasked, computed as by the wide kernel; the tree kernel's
             // workgroups take only the (at most two) splits holding the
             // tree's rows; both sets in one launch
             static_assert(64 + 1 <= SPLIT, "a tree (at most 64 nodes) spans at most two splits");
             AttnArgs lin = aa;
             lin.tree = 0;
             lin.split_mode = 1;
             AttnArgs tail = aa;
             tail.split_mode = 2;
             const int ty = std::min(nsplit, 2), tz = B * ((nqt + qt - 1) / qt);
             // query-tile groups of the wide part: as many as keep the whole
             // grid within one workgroup per CU (each holds 140 KB of LDS),
             // counting one split's worth of tree workgroups (the second
             // exits unless the tree's rows cross a split boundary)
             const int per = m.Hkv * nsplit * B;
             const int nqg = std::max(1, std::min((nqt + 7) / 8, (256 - m.Hkv * tz) / per));
             hipLaunchKernelGGL((attn_tree_wide_kernel<DT, HD>), dim3(m.Hkv * (ty * tz + nsplit * B * nqg)),
                                dim3(WIDE_THREADS), 0, st, tail, lin, nqg, ty, tz, nsplit);
             return last();
           }
           if (!aa.tree && wide) {
             // many query tiles: stage each split once per group of them; the
             // groups per sequence keep about two workgroups per CU in flight
             const int per = m.Hkv * nsplit * B;
             const int nqg = std::max(1, std::min((nqt + 7) / 8, (512 + per - 1) / per));
             hipLaunchKernelGGL((attn_wide_kernel<DT, HD>), dim3(m.Hkv, nsplit, B * nqg), dim3(WIDE_THREADS), 0, st,
                                aa, nqg);
             return last();
           }
           const dim3 grid(m.Hkv, nsplit, B * ((nqt + qt - 1) / qt));
           if (aa.tree)
             hipLaunchKernelGGL((attn_kernel<DT, HD, true>), grid, dim3(att_threads(true)), 0, st, aa);
           else
             hipLaunchKernelGGL((attn_kernel<DT, HD, false>), grid, dim3(att_threads(false)), 0, st, aa);
           return last();
         })) != hipSuccess)
      return e;
    if ((e = timed(prof, PC_COMBINE, st, [&] {
           constexpr int per_wg = CMB_THREADS * 4 / HD;   // (row, head) columns per workgroup
           static_assert(per_wg >= 1, "one column per workgroup at least");
           hipLaunchKernelGGL((attn_combine_kernel<DT, HD>), dim3((R * m.H + per_wg - 1) / per_wg), dim3(CMB_THREADS), 0,
                              st, w.attn_part,
                              w.info, nsplit, m.Hkv, G, R * G, m.H, T, (void*)w.xbuf, Sq);
           return last();
         })) != hipSuccess)
      return e;
    if (s.cap && (e = cap(l, c_o, w.xbuf, R16 * qdim * ESZ)) != hipSuccess) return e;
    // O projection; residual add + FFN norm (in the projection's epilogue when
    // fused: x = h * gain into x2buf and tile sums of h^2, else a kernel of
    // their own writing xbuf and chunk sums)
    if (fused) {
      EpArgs oa{};
      oa.w = lp.wo; oa.x = w.xbuf; oa.S = Sq; oa.n_tiles = d / 16; oa.n_items = d / 16;
      oa.d = d; oa.eps = m.eps; oa.h = w.h; oa.gain = lp.ffn_gain; oa.xout = (void*)w.x2buf; oa.x_S = Sd;
      oa.ssqt = w.ssqt;
      if ((e = timed(prof, PC_OPROJ, st, [&] { return gemm_ep<DT, EP_RESID>(oa, R, st); })) != hipSuccess) return e;
      if (s.cap && (e = cap(l, c_xf, w.x2buf, R16 * d * ESZ)) != hipSuccess) return e;
    } else {
    if ((e = timed(prof, PC_OPROJ, st, [&] { return gemm<DT>(lp.wo, w.xbuf, d, qdim, R, w.part, st); })) != hipSuccess)
      return e;
    if ((e = timed(prof, PC_NORM, st, [&] {
           hipLaunchKernelGGL((resid_kernel<DT, 1>), dim3((d + RES_COLS - 1) / RES_COLS, R), dim3(RES_THREADS), 0,
                              st, nullptr, nullptr, w.h, w.part, sk_q, R, lp.ffn_gain, d, (void*)w.xbuf, Sd, w.ssq);
           return last();
         })) != hipSuccess)
      return e;
    if (s.cap && (e = cap(l, c_xf, w.xbuf, R16 * d * ESZ)) != hipSuccess) return e;
    }
    // gate/up projection and SwiGLU: fused for d / KS <= FK_MAX_S, else
    // split-K partials and a SwiGLU launch
    if (fused_swiglu(d, DT)) {
      if ((e = timed(prof, PC_GATEUP, st, [&] {
             return fused ? gemm_swiglu<DT>(lp.wgu, w.x2buf, m.F, d, R, (void*)w.zbuf, w.ssq, w.ssqt, m.eps, st)
                          : gemm_swiglu<DT>(lp.wgu, w.xbuf, m.F, d, R, (void*)w.zbuf, w.ssq, nullptr, m.eps, st);
           })) != hipSuccess)
        return e;
    } else {
      if ((e = timed(prof, PC_GATEUP, st, [&] { return gemm<DT>(lp.wgu, w.xbuf, 2 * m.F, d, R, w.part, st); })) !=
          hipSuccess)
        return e;
      if ((e = timed(prof, PC_FINISH, st, [&] {
             hipLaunchKernelGGL((swiglu_kernel<DT>), dim3((m.F / 8 + 255) / 256, R), dim3(256), 0, st, w.part, sk_d,
                                R, m.F, (void*)w.zbuf, Sf, w.ssq, d, m.eps);
             return last();
           })) != hipSuccess)
        return e;
    }
    if (s.cap && (e = cap(l, c_z, w.zbuf, R16 * m.F * ESZ)) != hipSuccess) return e;
    // down projection; residual add + the next norm (layer l+1 attention side, or final)
    if ((e = timed(prof, PC_DOWN, st, [&] { return gemm<DT>(lp.wd, w.zbuf, d, m.F, R, w.part, st); })) != hipSuccess)
      return e;
    const float* gn = (l + 1 < m.L) ? m.layers[l + 1].attn_gain : m.final_gain;
    if ((e = timed(prof, PC_NORM, st, [&] {
           hipLaunchKernelGGL((resid_kernel<DT, 1>), dim3((d + RES_COLS - 1) / RES_COLS, R), dim3(RES_THREADS), 0,
                              st, nullptr, nullptr, w.h, w.part, sk_f, R, gn, d, (void*)w.xbuf, Sd, w.ssq);
           return last();
         })) != hipSuccess)
      return e;
    // x_attn of the next layer, or (after the last layer) x_final
    if (s.cap && (e = cap(l + 1, 0, w.xbuf, R16 * d * ESZ)) != hipSuccess) return e;
  }
  // LM head (without K slices when its reduction fits one workgroup), logits
  // + chunk maxima, argmax
  const bool lm1 = lm_head_one_slice(d, DT);
  if ((e = timed(prof, PC_LMHEAD, st, [&] {
         if (!lm1) return gemm<DT>(m.lm_head, w.xbuf, m.V, d, R, w.part, st);
         EpArgs la{};
         la.w = m.lm_head; la.x = w.xbuf; la.S = Sd; la.n_tiles = m.V / 16; la.n_items = m.V / 16; la.y = w.part;
         return gemm_ep<DT, EP_STORE>(la, R, st);
       })) != hipSuccess)
    return e;
  const int sk_lm = lm1 ? 1 : sk_d;
  const int nchunk = (m.V + 2047) / 2048;
  const bool topk = s.mode == 3;
  if ((e = timed(prof, PC_FINISH, st, [&] {
         if (topk)
           hipLaunchKernelGGL(logits_kernel<true>, dim3(nchunk, R), dim3(256), 0, st, w.part, sk_lm, R, m.V,
                              w.logits, w.amax, nchunk, w.ssq, d, m.eps);
         else
           hipLaunchKernelGGL(logits_kernel<false>, dim3(nchunk, R), dim3(256), 0, st, w.part, sk_lm, R, m.V,
                              w.logits, w.amax, nchunk, w.ssq, d, m.eps);
         return last();
       })) != hipSuccess)
    return e;
  return timed(prof, PC_ARGMAX, st, [&] {
    if (topk)
      hipLaunchKernelGGL(topk_select_kernel, dim3(R), dim3(64), 0, st, w.amax, nchunk, w.tok, w.info, s.T,
                         w.greedy, w.verdict);
    else if (s.mode == 4)
      hipLaunchKernelGGL(sample_stats_kernel, dim3(R), dim3(256), 0, st, w.logits, w.amax, nchunk, m.V, w.tok, s.T,
                         w.eps, w.sparam, w.rowstat, w.ebuf, w.greedy, w.verdict);
    else
      hipLaunchKernelGGL(argmax_kernel, dim3(R), dim3(256), 0, st, w.amax, nchunk, w.greedy);
    return last();
  });
}

// ------------------------------------------------------------ host staging --
//
// The per-call inputs are read straight from pinned host memory and the
// result records written straight back to it by kernels of the block itself,
// so a block waits on no copy-engine transfer before its first kernel or
// after its last.

__global__ __launch_bounds__(256) void stage_in_kernel(StageCopy sc) {
  int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= sc.total) return;
  int r = 0;
  while (r + 1 < sc.n && i >= sc.len[r]) i -= sc.len[r++];
  sc.dst[sc.off[r] + i] = sc.src[sc.off[r] + i];
}

__global__ __launch_bounds__(256) void result_out_kernel(const int* __restrict__ src, int* dst, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = src[i];
  __threadfence_system();
}

hipError_t run_stage_in(const StageCopy& sc, hipStream_t st) {
  if (sc.total <= 0) return hipSuccess;
  hipLaunchKernelGGL(stage_in_kernel, dim3((sc.total + 255) / 256), dim3(256), 0, st, sc);
  return hipGetLastError();
}

hipError_t run_result_out(const Work& w, int B, int* host_result, hipStream_t st) {
  const int n = B * w.rec;
  hipLaunchKernelGGL(result_out_kernel, dim3((n + 255) / 256), dim3(256), 0, st, w.result, host_result, n);
  return hipGetLastError();
}

hipError_t run_forward(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  if (m.dt == DT_BF16 && m.hd == 128) return forward_t<DT_BF16, 128>(m, w, s, prof, st);
  if (m.dt == DT_BF16 && m.hd == 64) return forward_t<DT_BF16, 64>(m, w, s, prof, st);
  if (m.dt == DT_F32 && m.hd == 64) return forward_t<DT_F32, 64>(m, w, s, prof, st);
  return hipErrorInvalidValue;
}

hipError_t run_accept(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  return timed(prof, PC_ACCEPT, st, [&] {
    hipLaunchKernelGGL(accept_kernel, dim3(s.B), dim3(64), 0, st, w.tok, w.prow, w.greedy, w.verdict, s.T,
                       s.mode, w.result, w.rec);
    if (s.mode == 4)   // one sequence: draw the next token at the accepted length
      hipLaunchKernelGGL(resample_kernel, dim3(1), dim3(256), 0, st, w.ebuf, m.V, w.tok, s.T, w.unif, w.sparam,
                         w.rowstat, w.result);
    return hipGetLastError();
  });
}

hipError_t run_gemm_sequence(const Model& m, const Work& w, int which, int R, hipStream_t st) {
  const int d = m.d, qdim = m.H * m.hd, qkvN = qdim + 2 * m.Hkv * m.hd;
  for (int l = 0; l < m.L; ++l) {
    const LayerPtrs& lp = m.layers[l];
    hipError_t e = hipErrorInvalidValue;
    const bool bf = m.dt == DT_BF16;
    const bool fused = fused_proj(d, qdim, m.hd, m.dt);
    const int ks = ks_of(m.dt);
    EpArgs ea{};
    ea.d = d; ea.eps = m.eps;
    if (which == PC_QKV) {
      // no K/V stores (the staged slots may hold committed rows)
      ea.w = lp.wqkv; ea.x = w.xbuf; ea.S = d / ks; ea.n_tiles = qkvN / 16; ea.n_items = qkvN / 32;
      ea.ssq = w.ssq; ea.H = m.H; ea.Hkv = m.Hkv; ea.hd = m.hd; ea.pos = w.pos; ea.rope = m.rope;
      ea.rowslot = w.slot; ea.q = w.q;
    } else if (which == PC_OPROJ) {
      ea.w = lp.wo; ea.x = w.xbuf; ea.S = qdim / ks; ea.n_tiles = d / 16; ea.n_items = d / 16;
      ea.h = w.h; ea.gain = lp.ffn_gain; ea.xout = (void*)w.x2buf; ea.x_S = d / ks; ea.ssqt = w.ssqt;
    }
    switch (which) {
      case PC_QKV:
        if (fused) e = bf ? gemm_ep<DT_BF16, EP_ROPE>(ea, R, st) : gemm_ep<DT_F32, EP_ROPE>(ea, R, st);
        else e = bf ? gemm<DT_BF16>(lp.wqkv, w.xbuf, qkvN, d, R, w.part, st)
                    : gemm<DT_F32>(lp.wqkv, w.xbuf, qkvN, d, R, w.part, st);
        break;
      case PC_OPROJ:
        if (fused) e = bf ? gemm_ep<DT_BF16, EP_RESID>(ea, R, st) : gemm_ep<DT_F32, EP_RESID>(ea, R, st);
        else e = bf ? gemm<DT_BF16>(lp.wo, w.xbuf, d, qdim, R, w.part, st)
                    : gemm<DT_F32>(lp.wo, w.xbuf, d, qdim, R, w.part, st);
        break;
      case PC_GATEUP:
        if (fused)
          e = bf ? gemm_swiglu<DT_BF16>(lp.wgu, w.x2buf, m.F, d, R, (void*)w.zbuf, w.ssq, w.ssqt, m.eps, st)
                 : gemm_swiglu<DT_F32>(lp.wgu, w.x2buf, m.F, d, R, (void*)w.zbuf, w.ssq, w.ssqt, m.eps, st);
        else if (fused_swiglu(d, m.dt))
          e = bf ? gemm_swiglu<DT_BF16>(lp.wgu, w.xbuf, m.F, d, R, (void*)w.zbuf, w.ssq, nullptr, m.eps, st)
                 : gemm_swiglu<DT_F32>(lp.wgu, w.xbuf, m.F, d, R, (void*)w.zbuf, w.ssq, nullptr, m.eps, st);
        else
          e = bf ? gemm<DT_BF16>(lp.wgu, w.xbuf, 2 * m.F, d, R, w.part, st)
                 : gemm<DT_F32>(lp.wgu, w.xbuf, 2 * m.F, d, R, w.part, st);
        break;
      case PC_DOWN: e = bf ? gemm<DT_BF16>(lp.wd, w.zbuf, d, m.F, R, w.part, st)
                           : gemm<DT_F32>(lp.wd, w.zbuf, d, m.F, R, w.part, st); break;
      case PC_LMHEAD:
        if (lm_head_one_slice(d, m.dt)) {
          EpArgs la{};
          la.w = m.lm_head; la.x = w.xbuf; la.S = d / ks; la.n_tiles = m.V / 16; la.n_items = m.V / 16;
          la.y = w.part;
          e = bf ? gemm_ep<DT_BF16, EP_STORE>(la, R, st) : gemm_ep<DT_F32, EP_STORE>(la, R, st);
        } else {
          e = bf ? gemm<DT_BF16>(m.lm_head, w.xbuf, m.V, d, R, w.part, st)
                 : gemm<DT_F32>(m.lm_head, w.xbuf, m.V, d, R, w.part, st);
        }
        break;
      default: break;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t run_compact(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  const size_t layer_elems = (size_t)m.max_pages * 2 * m.Hkv * 64 * m.hd;
  const dim3 grid(m.L * m.Hkv, s.B), block(256);
  return timed(prof, PC_COMPACT, st, [&] {
    if (m.dt == DT_BF16 && m.hd == 128)
      hipLaunchKernelGGL((compact_kernel<DT_BF16, 128>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, w.info, m.Hkv, w.ptable_len, w.rec);
    else if (m.dt == DT_BF16 && m.hd == 64)
      hipLaunchKernelGGL((compact_kernel<DT_BF16, 64>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, w.info, m.Hkv, w.ptable_len, w.rec);
    else if (m.dt == DT_F32 && m.hd == 64)
      hipLaunchKernelGGL((compact_kernel<DT_F32, 64>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, w.info, m.Hkv, w.ptable_len, w.rec);
    else
      return hipErrorInvalidValue;   // fp32 with head_dim 128 would exceed the LDS staging size
    return hipGetLastError();
  });
}

}  // namespace ee
