// da_internal.hpp -- launch arguments and plan shared by the C-ABI layer and
// the gfx950 kernels.  Not part of the public interface.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "delta_attn.h"

namespace da {

// Keys per tile of every attention kernel, and query rows per wavefront.
constexpr int kKeyTile = 64;
constexpr int kRowsPerWave = 32;
// Attention workgroups: kAttnWaves wavefronts share every K/V tile, which
// passes through a ring of kAttnStages LDS buffers (prefetch distance
// kAttnStages - 1 tiles).
constexpr int kAttnWaves = 8;
constexpr int kAttnStages = 2;
constexpr int kAttnThreads = 64 * kAttnWaves;
// Delta epilogue workgroups.
constexpr int kEpiThreads = 256;

// Division by a divisor fixed for a launch, for numerators below 2^31.  With
// l = ceil(log2 d) and m = floor(2^(31+l) / d) + 1 < 2^32, floor(x / d) =
// floor(x m / 2^(31+l)) for every 0 <= x < 2^31 (Granlund and Montgomery,
// "Division by invariant integers using multiplication", 1994, Thm. 4.2 with
// N = 31).  A uniform numerator costs three scalar instructions instead of
// a division routine.
struct FastDiv {
  uint32_t m;
  uint32_t sh;  // 31 + l
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while (l < 32 && (1ull << l) < d) ++l;
  FastDiv f;
  f.m = (uint32_t)(((1ull << (31 + l)) / d) + 1);
  f.sh = 31 + l;
  return f;
}

__host__ __device__ __forceinline__ uint32_t fdiv(uint32_t x, FastDiv f) {
  return (uint32_t)(((uint64_t)x * f.m) >> f.sh);
}

// Everything a kernel needs; passed by value as the kernel argument.
struct Args {
  const uint16_t* q;  // [T, Hq, d] bf16
  const uint16_t* k;  // [T, Hkv, d] bf16
  const uint16_t* v;  // [T, Hkv, d] bf16
  uint16_t* out;      // [T, Hq, d] bf16
  const int32_t* cu;  // device cu_seqlens [B+1], or nullptr for B sequences of N tokens
  int B, N;           // N: the fixed length, or max_seqlen when cu != nullptr
  int Hq, Hkv, d;
  int window, n_sink, gamma;
  float scale_log2;   // log2(e) / sqrt(d): scores are exponentiated with exp2
  // Anchors a < cover have a sparse key set equal to [0, a], so Delta = 0 there
  // and their groups keep the sparse rows: n_sink + window for sink + window
  // attention, 0 for key-block lists.
  int64_t cover;

  // Sparse attention from key-block lists (nullptr: sink + window).  Lists are
  // CSR per (sequence, kv head, query block of block_q rows): blk_ptr
  // [B][Hkv][nqb + 1] offsets into blk_idx (key tiles of kKeyTile keys).
  const int32_t* blk_ptr;
  const int32_t* blk_idx;
  int block_q, nqb;

  // Workgroup tiling of (query heads x rows): hpw heads of one kv group, each
  // with ppw sub-tiles of 32 rows; hpw * ppw == kAttnWaves.
  int hpw, ppw;
  int n_hgroups;      // Hq / hpw
  int n_rtiles;       // row tiles (of 32 * ppw rows) per (sequence, head group)
  // the launch's divisors: row tiles, key chunks, sequences, GQA group size
  // Hq / Hkv, gamma, query block
  FastDiv fd_rtiles, fd_nC, fd_B, fd_G, fd_gamma, fd_bq;
  // Dense-row workgroup order when every sequence has the same length (set by
  // launch_dense_rows; dr_n1 = 0 keeps the plain order).  Row tiles
  // [dr_t[c], dr_nrt) take the whole of key chunk c, [dr_z[c], dr_t[c]) part
  // of it, lower ones none.  The dr_n1 whole-chunk (row tile, chunk) pairs run
  // first, chunk by chunk, then the dr_n2 partial ones.
  int dr_n1, dr_n2, dr_nrt;
  int dr_t[16], dr_z[16];

  // Workspace of the Delta path (nullptr for the plain attention calls).
  float* sa;          // [B][Hq][nA_max][d]      sparse output at anchor rows, fp32
  float* dense;       // [B][Hq][nR_max][d]      merged dense rows, fp32 (fused schedule;
                      //                          the same memory as sa)
  float* part_o;      // [B][Hq][nR_max][nC][d]  unnormalised partial outputs of dense rows
  float* part_ml;     // [B][Hq][nR_max][nC][2]  (running max * scale_log2, normaliser)
  int nA_max;         // max anchors per sequence: floor(max_seqlen / gamma)
  int nR_max;         // max dense rows per sequence (anchors + tail rows)
  int nC;             // key chunks per dense row (split of the key axis)
  int chunk;          // keys per chunk, a multiple of kKeyTile
  int head_chunk;     // query heads per epilogue workgroup

  // Correction variants of step 5 (see delta_attn_prefill_correction).
  int corr_mode;      // DA_CORR_*
  float corr_p[3];    // EMA weight / filter coefficients
  float* dbuf;        // [B][Hq][nA_max][d]  Delta_i (filtered in place by the filter mode)
  float* ebuf;        // [B][Hq][nA_max][d]  EMA value entering group i

  // Fused schedule: the sparse kernel stores the corrected rows itself from the
  // merged dense rows (0: plain sparse store; 1: Delta correction; 2: recompute).
  int fuse;
};

// Sizes of the Delta path's workspace for a problem; all in elements/bytes.
struct Plan {
  int nA_max, nR_max, nC, chunk;
  size_t sa_floats, part_o_floats, part_ml_floats;  // sa: nR_max rows per (sequence, head)
  size_t bytes;
};

bool make_plan(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma, Plan* p,
               size_t limit = 0);

// The allocation-free entry point's workspace: a static device array of
// kScratchBytes (da_kernels.hip).  scratch_address gives its address on
// device `dev`, which must be the current device; it is looked up once per
// device and kept.
constexpr size_t kScratchBytes = DA_NOALLOC_SCRATCH_BYTES;
hipError_t scratch_address(int dev, void** p);
// Extra workspace floats the correction variants need beyond the plan.
size_t correction_floats(int B, int max_seqlen, int Hq, int d, int gamma, int mode);
int heads_per_block(int G);
// Heads per workgroup of the fused sparse kernel: the largest power of two
// dividing G (at most kAttnWaves) whose per-head row slab, 32 * kAttnWaves /
// hpw rows, is a multiple of gamma and at most max_rows; 0 when there is none.
int fused_heads_per_block(int G, int gamma, int max_rows);

// Kernel launchers (da_kernels.hip).  Each returns the hipError_t of the launch.
hipError_t launch_sparse(const Args& a, hipStream_t s);
hipError_t launch_dense(const Args& a, hipStream_t s);
hipError_t launch_dense_rows(const Args& a, hipStream_t s);
hipError_t launch_delta_epilogue(const Args& a, hipStream_t s);
hipError_t launch_correction(const Args& a, hipStream_t s);
hipError_t launch_check_inputs(const int32_t* cu, int B, int max_seqlen, const int32_t* bptr,
                              const int32_t* bidx, int64_t nnz, int Hkv, int nqb,
                              int32_t* result, hipStream_t s);

}  // namespace da
