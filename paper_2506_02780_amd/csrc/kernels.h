// Internal launch interface between the host engine (engine.cpp) and the
// gfx950 kernels (kernels.hip).  Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ee {

enum Dt { DT_F32 = 0, DT_BF16 = 1 };

// Fragment geometry shared by the weight packer, the GEMM and the producers
// of GEMM inputs.  One "fragment" is 16 bytes per lane of a 64-lane wave and
// covers 16 rows x KS columns of a matrix: lane (grp = lane / 16, col =
// lane % 16) holds row `col`, columns [s*KS + grp*KS/4, s*KS + grp*KS/4 +
// KS/4) of super-step s.  KS = 32 for bf16 (one 16x16x32 MFMA), 16 for fp32
// (four 16x16x4 MFMAs).
inline int ks_of(int dt) { return dt == DT_BF16 ? 32 : 16; }
inline int esz_of(int dt) { return dt == DT_BF16 ? 2 : 4; }

struct PackSrc {
  const void* src;   // logical row-major [rows, K]
  int rows;          // rows copied (multiple of 16)
  int dst_row0;      // first destination row (multiple of 16)
};

// Pack a logical matrix into the fragment layout
// dst[((tile * S + s) * 64 + lane) * 16 bytes], S = K / KS.
hipError_t launch_pack(const PackSrc& ps, void* dst, int K, int dt, hipStream_t st);

// K-slices of the split-K GEMM for a reduction length K (depends on K only).
int gemm_slices_for(int K, int dt);

// Copy/convert small arrays used as-is (embedding rows, gains).
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t st);

struct LayerPtrs {
  const uint4* wqkv;   // packed [(H + 2 Hkv) * hd, d]: q rows, k rows, v rows
  const uint4* wo;     // packed [d, H * hd]
  const uint4* wgu;    // packed [2F, d]: gate rows, then up rows
  const uint4* wd;     // packed [d, F]
  const float* attn_gain;
  const float* ffn_gain;
};

struct Model {
  int L, d, H, Hkv, hd, F, V, dt;
  float eps;
  int max_ctx, max_pages;   // pages per layer in the pool
  const void* embed;        // [V, d] row-major, model dtype
  const uint4* lm_head;     // packed [V, d]
  const float* final_gain;
  LayerPtrs* layers;        // host array of L
  void* kv_pool;            // [L][pages][2][Hkv][64 * hd]
  const float2* rope;       // [max_ctx][hd / 2] (cos, sin)
};

// Per-step device buffers (all inside the caller's workspace).  A block holds
// B sequences of T rows each, R = B * T rows in all (row b*T + t is row t of
// sequence b); Rmax = max_seqs * (k_max + 1).
struct Work {
  float* h;                 // [Rmax, d] residual stream
  float* ssq;               // [Rmax, 8] sums of h^2 over 1024-column chunks (the norms' row scales)
  uint4* xbuf;              // packed activations, max(d, H*hd) columns
  uint4* x2buf;             // packed activations, d columns (the FFN-side norm's output when
                            // the O projection applies the residual and norm itself)
  float* ssqt;              // [Rmax, d / 16] sums of h^2 per 16-column tile (that norm's row scales)
  uint4* zbuf;              // packed activations, F columns
  void* q;                  // [Rmax, H, hd] model dtype
  float* attn_part;         // [splits][Hkv][Rmax*G][hd + 2]
  float* part;              // GEMM slice partials [SK][R][N]
  float* logits;            // [Rmax, V]
  unsigned long long* amax; // [Rmax, ceil(V/2048), 8] chunk maxima (top-8 in mode 3)
  int* greedy;              // [Rmax]
  int* verdict;             // [Rmax] modes 3, 4: tau | draft-accepted << 8
  double* rowstat;          // [Rmax][2] mode 4: row maximum and sum of exp((l - max) / temperature)
  double* ebuf;             // [Rmax][V] mode 4: exp((l - max) / temperature) of every logit
  int* result;              // [max_seqs][rec]: accept_len, next, accepted rows (or thresholds)
  // staged per call (host -> device)
  int* tok;                 // [Rmax]
  int* pos;                 // [Rmax] rotary position of each row
  int* prow;                // [Rmax] parent row within the sequence (tree) or t-1
  int* slot;                // [Rmax] KV-pool slot (page * 64 + offset) the row's K/V go to
  unsigned char* path;      // [Rmax][64] tree mode (at most 64 nodes): entry j-1 of row t =
                            // block row at depth j on t's path (row 0, the pending token, is depth 0)
  int* ptable;              // [max_seqs][ptable_len] page of each 64-position block
  float* eps;               // [Rmax] mode 4: acceptance draws of the draft rows
  float* unif;              // [Rmax] mode 4: resampling draws (row a of the block)
  const unsigned char* sparam;  // mode 4: {u64 draft distribution pointer or 0, f32 temperature, i32 residual}
  int* info;                // [max_seqs][4]: committed positions n, attention splits in use,
                            // top-k size k and dynamic flag (mode 3)
  int ptable_len;           // entries per sequence (multiple of 4)
  int rec;                  // ints per result record: 2 + k_max
  int max_splits;           // attention splits of the longest context
};

// Optional per-launch timing: events recorded around launches of the classes
// selected in `mask` (bit = EE_PROF_* class).
struct Prof {
  uint32_t mask = 0;
  hipEvent_t* ev = nullptr;   // pairs: ev[2i] before, ev[2i+1] after launch i
  int* cls = nullptr;         // class of launch i
  int cap = 0;                // pairs available
  int used = 0;               // pairs recorded in the current block
  bool overflow = false;      // a block had more timed launches than pairs
  bool on(int c) const { return (mask >> c) & 1u; }
};

// Timed launch scopes of one block, at most: per layer QKV, rotary + KV
// append, attention, split merge, O, norm, gate/up, SwiGLU (unfused), down,
// norm; then the first norm, LM head, logits, selection, acceptance and tree
// compaction.
inline int prof_pairs_per_block(int n_layers) { return 10 * n_layers + 6; }

// Launch shape of one block.  Everything that changes from step to step
// (committed lengths, split counts, tokens, positions, pages) is read by the
// kernels from the staging block, so a captured graph of a (T, B, mode)
// shape can be replayed for any step.
struct Step {
  int T;        // rows per sequence
  int B;        // sequences in the block
  int mode;     // 0 prefill, 1 linear verify, 2 tree verify, 3 linear top-k verify,
                // 4 linear stochastic verify (one sequence)
  int splits;   // attention splits of the grid: the most any sequence of the
                // block uses, ceil((n + T) / 256); 1 .. max_splits
  unsigned char* cap = nullptr;   // test aid: copies of every rounding site's
                                  // values (capture_bytes(m, T * B) bytes), or null
};

// Bytes of a rounding-site capture of R rows (layout in ee_capture's contract).
size_t capture_bytes(int L, int d, int qdim, int kvdim, int F, int dt, int R);

enum ProfClass {
  PC_NORM = 0, PC_QKV, PC_ATTN, PC_COMBINE, PC_OPROJ, PC_GATEUP, PC_DOWN, PC_LMHEAD, PC_ARGMAX,
  PC_ACCEPT, PC_COMPACT, PC_FINISH, PC_N
};

// Word ranges copied from the pinned host mirror of the staging block into the
// device staging block by the first kernel of a block (the same word offsets
// on both sides).
struct StageCopy {
  const uint32_t* src;      // host mirror (device-visible address)
  uint32_t* dst;            // device staging block
  int n;                    // ranges in use
  int off[10], len[10];     // word offset and word count of each range
  int total;                // sum of the word counts
};
hipError_t run_stage_in(const StageCopy& sc, hipStream_t st);
// The result records of B sequences (B * rec ints) copied from the device to
// pinned host memory (device-visible address) by the last kernel of a block.
hipError_t run_result_out(const Work& w, int B, int* host_result, hipStream_t st);

hipError_t run_forward(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st);
hipError_t run_accept(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st);
hipError_t run_compact(const Model& m, const Work& w, const Step& s, Prof* prof, hipStream_t st);
// One streaming read of `bytes` (a multiple of 16) at `buf`; `sink` is one
// writable word (measurement aid).
hipError_t run_stream_read(const void* buf, size_t bytes, unsigned* sink, hipStream_t st);
// The GEMM of projection `which` (PC_QKV, PC_OPROJ, PC_GATEUP or PC_DOWN) for
// every layer in turn, or the LM head's (PC_LMHEAD) as many times, on R rows
// of the current activation buffers (timing).
hipError_t run_gemm_sequence(const Model& m, const Work& w, int which, int R, hipStream_t st);

}  // namespace ee
