// gfx950 kernels of the greedy speculative-verification step.
//
// One verify step runs the target model over a block of T <= 65 rows (the
// pending token plus up to 64 draft tokens, Eq. 3), decodes every row
// greedily and accepts the longest matching draft prefix (Eq. 7).  Weight
// streaming dominates: every linear layer is a skinny GEMM with T rows, so
// each weight byte is read once per step and the GEMMs are HBM-bound.
//
// Arithmetic layout (identical for every T, so a row's result never depends
// on how many other rows share its block; a K = 0 step and a K = 64 step give
// bitwise-equal rows):
//   * GEMM: weights are the MFMA A operand (16 output features per tile),
//     activations the B operand (16 rows per t-tile).  One workgroup owns one
//     16-feature tile over the whole reduction dimension; its KW waves take
//     super-steps round-robin and are summed in wave order.
//   * Attention: keys in splits of 256 absolute positions, each split in
//     64-position sub-tiles combined by an online softmax in order; splits
//     merged in order by a second kernel.
//   * Residual stream, accumulators, softmax and logits are fp32; bf16 models
//     round the norm outputs, q/k after rotary, v, the attention output and
//     the SwiGLU product to bf16 (nearest-even).

#include "kernels.h"

#include <hip/hip_runtime.h>
#include <math.h>

namespace ee {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte load (weights are read once per step).
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// ---------------------------------------------------------------- numerics --

__device__ __forceinline__ uint32_t f2bf_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;   // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                        // nearest, ties to even
  return u >> 16;
}
__device__ __forceinline__ float bf2f(uint32_t b) { return __uint_as_float(b << 16); }

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

// Destination row r of a packed layer -> source row, per RowMap.
__device__ __forceinline__ int map_row(int map, int r, int hd, int* sel) {
  *sel = 0;
  if (map == ROWS_IDENTITY) return r;
  const int tile = r >> 4, rr = r & 15, grp = rr >> 2, q = rr & 3;
  if (map == ROWS_ROPE) {
    // rows of head h: tile j of the head holds pairs i = 8j + 2grp + (q & 1),
    // rows q = 0,1 the first half, q = 2,3 the partner i + hd/2.
    const int tiles_per_head = hd >> 4;
    const int head = tile / tiles_per_head, j = tile % tiles_per_head;
    const int i = 8 * j + 2 * grp + (q & 1);
    return head * hd + i + ((q >> 1) ? (hd >> 1) : 0);
  }
  // ROWS_SWIGLU: tile j holds features f = 8j + 2grp + (q & 1); q = 0,1 gate, 2,3 up
  *sel = q >> 1;
  return 8 * tile + 2 * grp + (q & 1);
}

template <int DT>
__global__ void pack_kernel(const void* __restrict__ src0, const void* __restrict__ src1,
                            int map, int rows_in_call, int dst_row0, int K, int hd,
                            uint4* __restrict__ dst) {
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL;
  const int S = K / KS;
  // one thread per destination lane-fragment (16 bytes)
  const size_t frags = (size_t)rows_in_call / 16 * S * 64;
  for (size_t f = blockIdx.x * (size_t)blockDim.x + threadIdx.x; f < frags;
       f += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(f & 63);
    const size_t ts = f >> 6;
    const int s = (int)(ts % S);
    const int tile_local = (int)(ts / S);
    const int grp = lane >> 4, c = lane & 15;
    const int r_local = tile_local * 16 + c;     // row within this call's block
    int sel;
    const int sr = map_row(map, r_local, hd, &sel);
    const void* src = sel ? src1 : src0;
    const int col0 = s * KS + grp * EPL;   // EPL elements = 16 bytes, 16-byte aligned
    const uint4 v = *reinterpret_cast<const uint4*>(reinterpret_cast<const unsigned char*>(src) +
                                                    ((size_t)sr * K + col0) * Geo<DT>::ESZ);
    const size_t dtile = (size_t)(dst_row0 / 16 + tile_local);
    dst[(dtile * S + s) * 64 + lane] = v;
  }
}

hipError_t launch_pack(const PackSrc& ps, void* dst, int K, int dt, int head_dim, hipStream_t st) {
  const int ks = ks_of(dt);
  if (K % ks || ps.rows % 16 || ps.dst_row0 % 16) return hipErrorInvalidValue;
  const size_t frags = (size_t)ps.rows / 16 * (K / ks) * 64;
  const int threads = 256;
  const size_t want = (frags + threads - 1) / threads;
  const int blocks = (int)(want < 65536 ? want : 65536);
  if (dt == DT_BF16)
    hipLaunchKernelGGL(pack_kernel<DT_BF16>, dim3(blocks), dim3(threads), 0, st, ps.src0, ps.src1,
                       ps.map, ps.rows, ps.dst_row0, K, head_dim, reinterpret_cast<uint4*>(dst));
  else
    hipLaunchKernelGGL(pack_kernel<DT_F32>, dim3(blocks), dim3(threads), 0, st, ps.src0, ps.src1,
                       ps.map, ps.rows, ps.dst_row0, K, head_dim, reinterpret_cast<uint4*>(dst));
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
  return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, st);
}

// -------------------------------------------------------------------- GEMM --

enum Epi { EPI_LOGITS = 0, EPI_RESIDUAL = 1, EPI_QKV = 2, EPI_SWIGLU = 3 };

struct GemmArgs {
  const uint4* w;       // packed weights, S super-steps per tile
  const uint4* x;       // packed activations (same S)
  int S;
  int T;
  int n_tiles;
  // epilogue outputs
  float* out;           // EPI_LOGITS: logits [T][N]; EPI_RESIDUAL: h [T][N]
  int N;
  unsigned long long* amax;  // EPI_LOGITS: [T][n_tiles]
  void* z;              // EPI_SWIGLU: packed activations of the down projection
  int z_S;
  // EPI_QKV
  void* q;              // [T][H][hd]
  void* kv_layer;       // pool base of this layer: [pages][2][Hkv][64*hd]
  const int* ptable;
  const int* pos;
  const float2* rope;
  int n;                // committed positions (block row r lands in slot n + r)
  int H, Hkv, hd;
};

// One workgroup = one 16-feature tile over the whole reduction dimension.
template <int DT, int MT, int KW, int EPI>
__global__ __launch_bounds__(KW * 64) void gemm_kernel(GemmArgs a) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int tile = blockIdx.x;
  const int c = lane & 15;
  const int S = a.S;
  const uint4* __restrict__ wp = a.w + (size_t)tile * S * 64 + lane;
  const uint4* __restrict__ xp = a.x + lane;

  bool rowok[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rowok[m] = (m * 16 + c) < a.T;

  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  constexpr int U = 4;
  const uint4 zero = make_uint4(0, 0, 0, 0);
  int s = wv;
  for (; s + (U - 1) * KW < S; s += U * KW) {
    uint4 wf[U];
    uint4 xf[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) wf[u] = ld_stream(wp + (size_t)(s + u * KW) * 64);
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m)
        xf[u][m] = rowok[m] ? xp[((size_t)m * S + s + u * KW) * 64] : zero;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[m] = mma<DT>(wf[u], xf[u][m], acc[m]);
  }
  for (; s < S; s += KW) {
    const uint4 wf = ld_stream(wp + (size_t)s * 64);
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const uint4 xf = rowok[m] ? xp[((size_t)m * S + s) * 64] : zero;
      acc[m] = mma<DT>(wf, xf, acc[m]);
    }
  }

  // Sum the KW partial tiles in wave order.
  __shared__ f32x4 red[KW][MT][64];
  __shared__ float tileY[MT * 16][17];   // [row t][feature within tile]
#pragma unroll
  for (int m = 0; m < MT; ++m) red[wv][m][lane] = acc[m];
  __syncthreads();
  for (int i = threadIdx.x; i < MT * 64; i += KW * 64) {
    const int m = i >> 6, ln = i & 63;
    f32x4 v = red[0][m][ln];
    for (int k = 1; k < KW; ++k) v += red[k][m][ln];
    const int t = m * 16 + (ln & 15), f0 = 4 * (ln >> 4);
    tileY[t][f0 + 0] = v[0];
    tileY[t][f0 + 1] = v[1];
    tileY[t][f0 + 2] = v[2];
    tileY[t][f0 + 3] = v[3];
  }
  __syncthreads();

  const int T = a.T;
  if (EPI == EPI_LOGITS) {
    for (int i = threadIdx.x; i < T * 16; i += KW * 64) {
      const int t = i >> 4, f = i & 15;
      a.out[(size_t)t * a.N + tile * 16 + f] = tileY[t][f];
    }
    for (int t = threadIdx.x; t < T; t += KW * 64) {
      unsigned long long best = 0;
      for (int f = 0; f < 16; ++f) {
        float v = tileY[t][f];
        uint32_t u = __float_as_uint(v);
        if ((u & 0x7fffffffu) > 0x7f800000u) continue;   // NaN never wins
        if ((u & 0x7fffffffu) == 0) u = 0;                // -0 ties with +0
        const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
        const unsigned long long key =
            ((unsigned long long)ord << 32) | (0xffffffffu - (uint32_t)(tile * 16 + f));
        best = key > best ? key : best;
      }
      a.amax[(size_t)t * a.n_tiles + tile] = best;
    }
  } else if (EPI == EPI_RESIDUAL) {
    for (int i = threadIdx.x; i < T * 16; i += KW * 64) {
      const int t = i >> 4, f = i & 15;
      a.out[(size_t)t * a.N + tile * 16 + f] += tileY[t][f];
    }
  } else if (EPI == EPI_SWIGLU) {
    // tile j, lane group grp, q: feature 8j + 2grp + (q & 1); q = 0,1 gate, q = 2,3 up
    for (int i = threadIdx.x; i < T * 8; i += KW * 64) {
      const int t = i >> 3, p = i & 7, grp = p >> 1, e = p & 1;
      const float gte = tileY[t][4 * grp + e], up = tileY[t][4 * grp + 2 + e];
      const float zv = gte / (1.0f + expf(-gte)) * up;
      const int f = 8 * tile + 2 * grp + e;
      store_elt<DT>(a.z, frag_index<DT>(t, f, a.z_S), zv);
    }
  } else {  // EPI_QKV
    const int hd = a.hd, half = hd >> 1;
    const int row0 = tile * 16;                       // packed row of this tile
    const int qrows = a.H * hd, krows = a.Hkv * hd;
    for (int i = threadIdx.x; i < T * 8; i += KW * 64) {
      const int t = i >> 3, p = i & 7, grp = p >> 1, e = p & 1;
      const int slot = a.n + t;
      const int page = a.ptable[slot >> 6], sp = slot & 63;
      if (row0 < qrows + krows) {
        // rotary pair: rows 4grp + e (first half) and 4grp + 2 + e (partner)
        const bool isq = row0 < qrows;
        const int base = isq ? row0 : row0 - qrows;
        const int head = base / hd, j = (base % hd) >> 4;
        const int di = 8 * j + 2 * grp + e;
        const float2 cs = a.rope[(size_t)a.pos[t] * half + di];
        const float x1 = tileY[t][4 * grp + e], x2 = tileY[t][4 * grp + 2 + e];
        const float y1 = x1 * cs.x - x2 * cs.y;
        const float y2 = x2 * cs.x + x1 * cs.y;
        if (isq) {
          const size_t qb = ((size_t)t * a.H + head) * hd;
          store_elt<DT>(a.q, qb + di, y1);
          store_elt<DT>(a.q, qb + di + half, y2);
        } else {
          const size_t kb = (((size_t)page * 2 + 0) * a.Hkv + head) * 64 * hd + (size_t)sp * hd;
          store_elt<DT>(a.kv_layer, kb + di, y1);
          store_elt<DT>(a.kv_layer, kb + di + half, y2);
        }
      } else {
        const int base = row0 - qrows - krows;
        const int head = base / hd, d0 = base % hd;
        // value rows are in natural order: tile row rr is dim d0 + rr; V stored [dim][slot]
        const size_t vb = (((size_t)page * 2 + 1) * a.Hkv + head) * 64 * hd;
        const int r1 = 4 * grp + e, r2 = 4 * grp + 2 + e;
        store_elt<DT>(a.kv_layer, vb + (size_t)(d0 + r1) * 64 + sp, tileY[t][r1]);
        store_elt<DT>(a.kv_layer, vb + (size_t)(d0 + r2) * 64 + sp, tileY[t][r2]);
      }
    }
  }
}

template <int DT, int EPI, int KW>
static hipError_t gemm_dispatch_mt(const GemmArgs& a, hipStream_t st) {
  const int mt = (a.T + 15) / 16;
  const dim3 grid(a.n_tiles), block(KW * 64);
  switch (mt) {
    case 1: hipLaunchKernelGGL((gemm_kernel<DT, 1, KW, EPI>), grid, block, 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<DT, 2, KW, EPI>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemm_kernel<DT, 3, KW, EPI>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<DT, 4, KW, EPI>), grid, block, 0, st, a); break;
    case 5: hipLaunchKernelGGL((gemm_kernel<DT, 5, KW, EPI>), grid, block, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int DT, int EPI>
static hipError_t gemm(const GemmArgs& a, hipStream_t st) {
  // waves per tile depend only on the reduction length, never on T
  if (a.S >= 256) return gemm_dispatch_mt<DT, EPI, 8>(a, st);
  if (a.S >= 64) return gemm_dispatch_mt<DT, EPI, 4>(a, st);
  return gemm_dispatch_mt<DT, EPI, 2>(a, st);
}

// ------------------------------------------------------------ embed / norm --

// Fixed-order block sum of one float per thread (blockDim.x == 256).
__device__ __forceinline__ float block_sum256(float v, float* sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) sh[threadIdx.x] = sh[threadIdx.x] + sh[threadIdx.x + w];
    __syncthreads();
  }
  const float r = sh[0];
  __syncthreads();
  return r;
}

// Row t: optionally h = E[tok[t]]; x = RMSNorm(h) * gain -> packed activation.
template <int DT, bool EMBED>
__global__ __launch_bounds__(256) void norm_kernel(const void* __restrict__ embed,
                                                   const int* __restrict__ tok, float* __restrict__ h,
                                                   const float* __restrict__ gain, float eps, int d,
                                                   void* __restrict__ xout, int x_S) {
  __shared__ float sh[256];
  const int t = blockIdx.x;
  float* hr = h + (size_t)t * d;
  if (EMBED) {
    const size_t e0 = (size_t)tok[t] * d;
    for (int i = threadIdx.x; i < d; i += 256) hr[i] = load_elt<DT>(embed, e0 + i);
  }
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float v = hr[i];
    ss = fmaf(v, v, ss);
  }
  ss = block_sum256(ss, sh);
  const float r = 1.0f / sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256)
    store_elt<DT>(xout, frag_index<DT>(t, i, x_S), hr[i] * r * gain[i]);
}

// --------------------------------------------------------------- attention --

struct AttnArgs {
  const void* q;            // [T][H][hd]
  const void* kv_layer;     // [pages][2][Hkv][64*hd]
  const int* ptable;
  const int* pos;
  const unsigned long long* anc;
  int T, n, H, Hkv, G, ncols;
  int tree;
  float scale_log2;         // log2(e) / sqrt(hd)
  float* part;              // [splits][Hkv][ncols][hd + 2]
};

constexpr int SPLIT = 256;  // keys per split (4 sub-tiles of 64)

template <int DT, int HD>
__global__ __launch_bounds__(1024) void attn_kernel(AttnArgs a) {
  constexpr int KS = Geo<DT>::KS, EPL = Geo<DT>::EPL, ESZ = Geo<DT>::ESZ;
  constexpr int NS = HD / KS;          // fragments along head_dim
  constexpr int ND = HD / 16;          // output dim tiles
  constexpr int ROWB = HD * ESZ;       // bytes of one key row
  constexpr int KROW = ROWB + 16;      // padded LDS row strides (bank spread)
  constexpr int VROW = 64 * ESZ + 16;
  __shared__ __attribute__((aligned(16))) unsigned char Ks[64 * KROW];
  __shared__ __attribute__((aligned(16))) unsigned char Vt[HD * VROW];

  const int sp = blockIdx.x, gkv = blockIdx.y, qgrp = blockIdx.z;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const int grp = lane >> 4, c = lane & 15;
  const int qt = qgrp * nw + wv;
  const int qc = qt * 16 + c;
  const bool colok = qc < a.ncols;
  const int t = colok ? qc / a.G : 0;
  const int head = gkv * a.G + (colok ? qc % a.G : 0);
  const int mypos = colok ? a.pos[t] : -1;
  const unsigned long long myanc = (colok && a.tree) ? a.anc[t] : 0ull;
  const int nkeys = a.n + a.T;          // slots written so far

  // query fragments (B operand): column qc, head dims [s*KS + grp*EPL, +EPL)
  uint4 qf[NS];
  {
    const unsigned char* qb =
        reinterpret_cast<const unsigned char*>(a.q) + ((size_t)t * a.H + head) * ROWB;
#pragma unroll
    for (int s = 0; s < NS; ++s)
      qf[s] = colok ? *reinterpret_cast<const uint4*>(qb + (s * KS + grp * EPL) * ESZ)
                    : make_uint4(0, 0, 0, 0);
  }

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o_run[ND];
#pragma unroll
  for (int i = 0; i < ND; ++i) o_run[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  const size_t head_stride = (size_t)64 * HD;   // elements per (page, kv, head) block
  for (int st = 0; st < SPLIT / 64; ++st) {
    const int base = sp * SPLIT + st * 64;
    if (base >= nkeys) break;
    const int page = a.ptable[base >> 6];
    const unsigned char* kg = reinterpret_cast<const unsigned char*>(a.kv_layer) +
                              ((((size_t)page * 2 + 0) * a.Hkv + gkv) * head_stride) * ESZ;
    const unsigned char* vg = reinterpret_cast<const unsigned char*>(a.kv_layer) +
                              ((((size_t)page * 2 + 1) * a.Hkv + gkv) * head_stride) * ESZ;
    const int valid = nkeys - base;    // keys in this sub-tile that were written
    // K rows [64][HD]: zero rows >= valid
    for (int i = threadIdx.x; i < 64 * ROWB / 16; i += blockDim.x) {
      const int row = i / (ROWB / 16), col = i % (ROWB / 16);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < valid) v = *reinterpret_cast<const uint4*>(kg + (size_t)i * 16);
      *reinterpret_cast<uint4*>(Ks + row * KROW + col * 16) = v;
    }
    // V^T [HD][64]: zero columns >= valid
    for (int i = threadIdx.x; i < HD * 64 * ESZ / 16; i += blockDim.x) {
      uint4 v = *reinterpret_cast<const uint4*>(vg + (size_t)i * 16);
      if (valid < 64) {
        const int col0 = ((i * 16) / ESZ) & 63;   // 16 bytes never straddle a dim row
        if (DT == DT_BF16) {
          uint32_t w[4] = {v.x, v.y, v.z, v.w};
          for (int e = 0; e < 8; ++e)
            if (col0 + e >= valid) w[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
          v = make_uint4(w[0], w[1], w[2], w[3]);
        } else {
          if (col0 + 0 >= valid) v.x = 0;
          if (col0 + 1 >= valid) v.y = 0;
          if (col0 + 2 >= valid) v.z = 0;
          if (col0 + 3 >= valid) v.w = 0;
        }
      }
      constexpr int VU = 64 * ESZ / 16;   // uint4 per V^T row
      *reinterpret_cast<uint4*>(Vt + (i / VU) * VROW + (i % VU) * 16) = v;
    }
    __syncthreads();

    // S^T = K Q^T for 4 key tiles of 16: lane holds key 16kt + 4grp + r, column c
    f32x4 sacc[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sacc[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4 kf = *reinterpret_cast<const uint4*>(Ks + (size_t)(16 * kt + c) * KROW +
                                                         (s * KS + grp * EPL) * ESZ);
        sacc[kt] = mma<DT>(kf, qf[s], sacc[kt]);
      }
    }
    float sv[4][4];
    float m_sub = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int kp = base + 16 * kt + 4 * grp + r;
        bool vis;
        if (!a.tree) {
          vis = kp <= mypos;
        } else {
          const int br = kp - a.n;   // block row held by this slot
          vis = colok && ((kp < a.n) || br == 0 ||
                          (br >= 1 && br < a.T && ((myanc >> (br - 1)) & 1ull)));
        }
        const float x = vis ? sacc[kt][r] * a.scale_log2 : -INFINITY;
        sv[kt][r] = x;
        m_sub = fmaxf(m_sub, x);
      }
    m_sub = fmaxf(m_sub, __shfl_xor(m_sub, 16));
    m_sub = fmaxf(m_sub, __shfl_xor(m_sub, 32));
    const float m_new = fmaxf(m_run, m_sub);
    const bool any = m_new != -INFINITY;
    const float alpha = (any && m_run != -INFINITY) ? exp2f(m_run - m_new) : (any ? 0.f : 1.f);
    float p[4][4];
    float l_sub = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        p[kt][r] = any ? exp2f(sv[kt][r] - m_new) : 0.f;
        l_sub += p[kt][r];
      }
    l_sub += __shfl_xor(l_sub, 16);
    l_sub += __shfl_xor(l_sub, 32);
    l_run = l_run * alpha + l_sub;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < ND; ++i) o_run[i] *= alpha;

    // O^T += V^T P^T; reduction over the 64 keys of the sub-tile
    if (DT == DT_BF16) {
      // P enters the bf16 MFMA as hi + lo bf16 parts (about 16 significant
      // bits), so the weights of the value rows keep near-fp32 precision.
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2) {
        uint32_t ph[8], pl[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = p[2 * k2 + (e >> 2)][e & 3];
          ph[e] = f2bf_bits(pv);
          pl[e] = f2bf_bits(pv - bf2f(ph[e]));
        }
        const uint4 pfh = make_uint4(ph[0] | (ph[1] << 16), ph[2] | (ph[3] << 16),
                                     ph[4] | (ph[5] << 16), ph[6] | (ph[7] << 16));
        const uint4 pfl = make_uint4(pl[0] | (pl[1] << 16), pl[2] | (pl[3] << 16),
                                     pl[4] | (pl[5] << 16), pl[6] | (pl[7] << 16));
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
          const unsigned char* vr = Vt + (size_t)(16 * dt + c) * VROW;
          const uint2 lo = *reinterpret_cast<const uint2*>(vr + (32 * k2 + 4 * grp) * ESZ);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + (32 * k2 + 16 + 4 * grp) * ESZ);
          const uint4 vf = make_uint4(lo.x, lo.y, hi.x, hi.y);
          o_run[dt] = mma<DT>(vf, pfh, o_run[dt]);
          o_run[dt] = mma<DT>(vf, pfl, o_run[dt]);
        }
      }
    } else {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        const uint4 pf = make_uint4(__float_as_uint(p[kt][0]), __float_as_uint(p[kt][1]),
                                    __float_as_uint(p[kt][2]), __float_as_uint(p[kt][3]));
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
          const unsigned char* vr = Vt + (size_t)(16 * dt + c) * VROW;
          const uint4 vf = *reinterpret_cast<const uint4*>(vr + (16 * kt + 4 * grp) * ESZ);
          o_run[dt] = mma<DT>(vf, pf, o_run[dt]);
        }
      }
    }
    __syncthreads();
  }

  if (colok) {
    float* out = a.part + (((size_t)sp * a.Hkv + gkv) * a.ncols + qc) * (HD + 2);
#pragma unroll
    for (int dt = 0; dt < ND; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) out[16 * dt + 4 * grp + r] = o_run[dt][r];
    if (grp == 0) {
      out[HD] = m_run;
      out[HD + 1] = l_run;
    }
  }
}

// Merge the splits of every (row, head) in split order; write the attention
// output as packed activations of the O projection.
template <int DT, int HD>
__global__ __launch_bounds__(HD) void attn_combine_kernel(const float* __restrict__ part, int nsplit,
                                                         int Hkv, int G, int ncols, int H,
                                                         void* __restrict__ xout, int x_S) {
  const int t = blockIdx.x / H, j = blockIdx.x % H;
  const int gkv = j / G, qc = t * G + (j % G);
  const int dim = threadIdx.x;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) {
    const float* p = part + (((size_t)s * Hkv + gkv) * ncols + qc) * (HD + 2);
    if (p[HD + 1] > 0.f) M = fmaxf(M, p[HD]);
  }
  float L = 0.f, O = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float* p = part + (((size_t)s * Hkv + gkv) * ncols + qc) * (HD + 2);
    const float l = p[HD + 1];
    if (!(l > 0.f)) continue;
    const float w = exp2f(p[HD] - M);
    L = fmaf(l, w, L);
    O = fmaf(p[dim], w, O);
  }
  store_elt<DT>(xout, frag_index<DT>(t, j * HD + dim, x_S), O / L);
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

// result[0] = accepted rows a, result[1] = next token, result[2..2+a) = accepted
// block rows in depth order.  Mode 0 (prefill) commits every row.
__global__ __launch_bounds__(64) void accept_kernel(const int* __restrict__ tok,
                                                    const int* __restrict__ prow,
                                                    const int* __restrict__ greedy, int T, int mode,
                                                    int* __restrict__ result) {
  const int lane = threadIdx.x;
  const int K = T - 1;
  if (mode == 0) {
    if (lane == 0) {
      result[0] = T - 1;
      result[1] = greedy[T - 1];
    }
    return;
  }
  if (mode == 1) {
    // draft d_{i+1} (row i+1) is checked against the greedy token of row i
    const bool mism = lane < K && tok[lane + 1] != greedy[lane];
    const unsigned long long b = __ballot(mism);
    const int a = b ? __ffsll((long long)b) - 1 : K;
    if (lane == 0) {
      result[0] = a;
      result[1] = greedy[a];
    }
    if (lane < a) result[2 + lane] = lane + 1;
    return;
  }
  // tree walk from row 0
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
                                                      const int* __restrict__ result, int n, int Hkv) {
  constexpr int ESZ = Geo<DT>::ESZ;
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

// Runs `launch` bracketed by profiling events when class `c` is selected.
template <typename F>
static hipError_t timed(Prof* prof, int c, hipStream_t st, F&& launch) {
  const bool on = prof && prof->on(c) && prof->used < prof->cap;
  hipError_t e;
  if (on && (e = hipEventRecord(prof->ev[2 * prof->used], st)) != hipSuccess) return e;
  if ((e = launch()) != hipSuccess) return e;
  if (on) {
    if ((e = hipEventRecord(prof->ev[2 * prof->used + 1], st)) != hipSuccess) return e;
    prof->cls[prof->used++] = c;
  }
  return hipSuccess;
}

template <int DT, int HD>
static hipError_t forward_t(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  constexpr int KS = Geo<DT>::KS;
  const int T = s.T, d = m.d, qdim = m.H * m.hd;
  const int Sd = d / KS, Sq = qdim / KS, Sf = m.F / KS;
  const size_t layer_elems = (size_t)m.max_pages * 2 * m.Hkv * 64 * m.hd;
  hipError_t e;
  auto last = [] { return hipGetLastError(); };

  if ((e = timed(prof, PC_NORM, st, [&] {
         hipLaunchKernelGGL((norm_kernel<DT, true>), dim3(T), dim3(256), 0, st, m.embed, w.tok, w.h,
                            m.layers[0].attn_gain, m.eps, d, (void*)w.xbuf, Sd);
         return last();
       })) != hipSuccess)
    return e;

  const int G = m.H / m.Hkv, ncols = T * G;
  const int nkeys = s.n + T;
  const int nsplit = (nkeys + SPLIT - 1) / SPLIT;
  const int nqt = (ncols + 15) / 16;
  const int nqg = (nqt + 15) / 16;
  const int wpb = (nqt + nqg - 1) / nqg;

  for (int l = 0; l < m.L; ++l) {
    const LayerPtrs& lp = m.layers[l];
    void* kvl = reinterpret_cast<unsigned char*>(m.kv_pool) + l * layer_elems * Geo<DT>::ESZ;
    GemmArgs g{};
    g.T = T;
    // QKV + rotary + KV append
    g.w = lp.wqkv; g.x = w.xbuf; g.S = Sd; g.n_tiles = (qdim + 2 * m.Hkv * m.hd) / 16;
    g.q = w.q; g.kv_layer = kvl; g.ptable = w.ptable; g.pos = w.pos; g.rope = m.rope; g.n = s.n;
    g.H = m.H; g.Hkv = m.Hkv; g.hd = m.hd;
    if ((e = timed(prof, PC_QKV, st, [&] { return gemm<DT, EPI_QKV>(g, st); })) != hipSuccess) return e;
    // attention
    AttnArgs aa{};
    aa.q = w.q; aa.kv_layer = kvl; aa.ptable = w.ptable; aa.pos = w.pos; aa.anc = w.anc;
    aa.T = T; aa.n = s.n; aa.H = m.H; aa.Hkv = m.Hkv; aa.G = G; aa.ncols = ncols;
    aa.tree = s.mode == 2;
    aa.scale_log2 = 1.4426950408889634f / sqrtf((float)m.hd);
    aa.part = w.attn_part;
    if ((e = timed(prof, PC_ATTN, st, [&] {
           hipLaunchKernelGGL((attn_kernel<DT, HD>), dim3(nsplit, m.Hkv, nqg), dim3(wpb * 64), 0, st, aa);
           return last();
         })) != hipSuccess)
      return e;
    if ((e = timed(prof, PC_COMBINE, st, [&] {
           hipLaunchKernelGGL((attn_combine_kernel<DT, HD>), dim3(T * m.H), dim3(HD), 0, st, w.attn_part,
                              nsplit, m.Hkv, G, ncols, m.H, (void*)w.xbuf, Sq);
           return last();
         })) != hipSuccess)
      return e;
    // O projection + residual
    g = GemmArgs{};
    g.T = T; g.w = lp.wo; g.x = w.xbuf; g.S = Sq; g.n_tiles = d / 16; g.out = w.h; g.N = d;
    if ((e = timed(prof, PC_OPROJ, st, [&] { return gemm<DT, EPI_RESIDUAL>(g, st); })) != hipSuccess) return e;
    // FFN norm
    if ((e = timed(prof, PC_NORM, st, [&] {
           hipLaunchKernelGGL((norm_kernel<DT, false>), dim3(T), dim3(256), 0, st, nullptr, nullptr, w.h,
                              lp.ffn_gain, m.eps, d, (void*)w.xbuf, Sd);
           return last();
         })) != hipSuccess)
      return e;
    // gate/up + SwiGLU
    g = GemmArgs{};
    g.T = T; g.w = lp.wgu; g.x = w.xbuf; g.S = Sd; g.n_tiles = 2 * m.F / 16; g.z = w.zbuf; g.z_S = Sf;
    if ((e = timed(prof, PC_GATEUP, st, [&] { return gemm<DT, EPI_SWIGLU>(g, st); })) != hipSuccess) return e;
    // down + residual
    g = GemmArgs{};
    g.T = T; g.w = lp.wd; g.x = w.zbuf; g.S = Sf; g.n_tiles = d / 16; g.out = w.h; g.N = d;
    if ((e = timed(prof, PC_DOWN, st, [&] { return gemm<DT, EPI_RESIDUAL>(g, st); })) != hipSuccess) return e;
    // next norm: attention side of layer l+1, or the final norm
    const float* gn = (l + 1 < m.L) ? m.layers[l + 1].attn_gain : m.final_gain;
    if ((e = timed(prof, PC_NORM, st, [&] {
           hipLaunchKernelGGL((norm_kernel<DT, false>), dim3(T), dim3(256), 0, st, nullptr, nullptr, w.h,
                              gn, m.eps, d, (void*)w.xbuf, Sd);
           return last();
         })) != hipSuccess)
      return e;
  }
  // LM head + argmax partials
  GemmArgs g{};
  g.T = T; g.w = m.lm_head; g.x = w.xbuf; g.S = Sd; g.n_tiles = m.V / 16; g.out = w.logits; g.N = m.V;
  g.amax = w.amax;
  if ((e = timed(prof, PC_LMHEAD, st, [&] { return gemm<DT, EPI_LOGITS>(g, st); })) != hipSuccess) return e;
  return timed(prof, PC_ARGMAX, st, [&] {
    hipLaunchKernelGGL(argmax_kernel, dim3(T), dim3(256), 0, st, w.amax, m.V / 16, w.greedy);
    return last();
  });
}

hipError_t run_forward(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  if (m.dt == DT_BF16 && m.hd == 128) return forward_t<DT_BF16, 128>(m, w, s, prof, st);
  if (m.dt == DT_BF16 && m.hd == 64) return forward_t<DT_BF16, 64>(m, w, s, prof, st);
  if (m.dt == DT_F32 && m.hd == 128) return forward_t<DT_F32, 128>(m, w, s, prof, st);
  if (m.dt == DT_F32 && m.hd == 64) return forward_t<DT_F32, 64>(m, w, s, prof, st);
  return hipErrorInvalidValue;
}

hipError_t run_accept(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  (void)m;
  return timed(prof, PC_ACCEPT, st, [&] {
    hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(64), 0, st, w.tok, w.prow, w.greedy, s.T, s.mode,
                       w.result);
    return hipGetLastError();
  });
}

hipError_t run_compact(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st) {
  const size_t layer_elems = (size_t)m.max_pages * 2 * m.Hkv * 64 * m.hd;
  const dim3 grid(m.L * m.Hkv), block(256);
  return timed(prof, PC_COMPACT, st, [&] {
    if (m.dt == DT_BF16 && m.hd == 128)
      hipLaunchKernelGGL((compact_kernel<DT_BF16, 128>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, s.n, m.Hkv);
    else if (m.dt == DT_BF16 && m.hd == 64)
      hipLaunchKernelGGL((compact_kernel<DT_BF16, 64>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, s.n, m.Hkv);
    else if (m.dt == DT_F32 && m.hd == 64)
      hipLaunchKernelGGL((compact_kernel<DT_F32, 64>), grid, block, 0, st, m.kv_pool, layer_elems, w.ptable, w.result, s.n, m.Hkv);
    else
      return hipErrorInvalidValue;   // fp32 with head_dim 128 would exceed the LDS staging size
    return hipGetLastError();
  });
}

}  // namespace ee
