// da_kernels.hip -- gfx950 (CDNA4) kernels of the Delta Attention prefill.
//
// Delta Attention (arXiv 2505.11254, Algorithm 1) runs three steps:
//   1. sparse attention A*V for every query (StreamingLLM sinks + window, or
//      key tiles from per-query-block lists for other sparse bases),
//   2. dense causal attention A~V for every gamma-th query row (Eq. 4),
//   3. Delta = A~V - (A*V) at those rows, added to the gamma rows each covers
//      (Eq. 6); rows after the last whole group are computed densely
//      (implementation-details appendix).
// Steps 1 and 2 and the dense causal baseline share one attention kernel
// template (`attn_kernel`); step 3 is `delta_epilogue_kernel`.  The fused
// schedule runs step 2 first, merges its dense rows, and lets the sparse
// kernel store sparse + Delta directly, which saves the in-place pass over
// the output.
//
// Tile core (one wavefront = 32 query rows, 64-key tiles, bf16 MFMA):
//   S^T[key][row] = K Q^T   with v_mfma_f32_32x32x16_bf16: A = K rows from
//                           LDS, B = the wave's Q rows held in registers;
//   P^T = exp2(S^T * log2(e)/sqrt(d) - m)   online softmax in fp32;
//   O^T[dim][row] += V^T P^T  A = V^T read from the row-major V tile with
//                           gfx950's transposing LDS reads, B = P^T taken
//                           straight from the S^T accumulator registers.
// With this orientation a lane owns one query row in every accumulator
// (lane % 32 = row), so the row max, the normaliser and the rescale of O
// stay in the lane apart from one exchange with lane ^ 32, and P never goes
// through LDS.  K/V tiles go through a ring of LDS buffers; the waves of a
// workgroup share every K/V tile between the query heads of one GQA group.
#include "da_internal.hpp"

#include <math.h>

#include <algorithm>
#include <atomic>

namespace da {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

enum Mode { kSparse = 0, kDense = 1, kDenseRows = 2 };
// Per-element masks of a partly visible key tile (tile classes 2..5).
enum MaskKind { kMaskCausal = 2, kMaskWindow = 3, kMaskBoth = 4, kMaskAll = 5 };

// LDS layout of one pipeline stage (bf16 elements): K and V tiles of 64 keys,
// both row-major [key][dim] with unpadded rows of 2*D bytes.  Tiles arrive by
// LDS DMA, which writes 1 KB contiguous per wave instruction, so bank
// conflicts are avoided by XOR-swizzling the 16-byte chunks of each row
// instead of padding it:
//   K: chunk c of key row r sits at c ^ kswz(r), which spreads the 16-byte
//      operand reads of 16 consecutive keys over all banks;
//   V: chunk c of key row r sits at c ^ vswz(r), which spreads the transposing
//      8-byte reads (four keys x sixteen dims per 16-lane group).
template <int D>
struct Lds {
  static constexpr int kElems = kKeyTile * D;
  static constexpr int vElems = kKeyTile * D;
  static constexpr int stageElems = kElems + vElems;
  static constexpr int kRegions = kKeyTile * D * 2 / 1024;  // 1 KB DMA regions per tile
  static constexpr int kRegionsPerWave = kRegions / kAttnWaves;
  __device__ static constexpr int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
  __device__ static constexpr int vswz(int r) {
    return D == 128 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
  }
};

struct Seq {
  int64_t base;  // first token row of the sequence
  int L;         // its length
};

__device__ __forceinline__ Seq seq_of(const Args& a, int b) {
  if (a.cu) {
    const int s0 = a.cu[b], s1 = a.cu[b + 1];
    return {s0, s1 - s0};
  }
  return {(int64_t)b * a.N, a.N};
}

// Workgroups are dispatched in order, round-robin over the 8 XCDs (block i ->
// XCD i % 8), each with its own L2.  Logical blocks are ordered head group
// outermost, then sequence, [key chunk,] row tile.
//  - When the head groups split evenly over the XCDs, XCD x takes the
//    contiguous eighth [x*n/8, (x+1)*n/8): whole head groups, each with every
//    sequence, so the XCDs get equal work and each streams its own kv heads'
//    keys and values through its L2 while neighbouring tiles share them.
//  - Otherwise XCD x takes the logical chunks x, x+8, x+16, ... of kXcdChunk
//    consecutive blocks: neighbouring tiles still run together on one L2,
//    and all XCDs walk the logical order at the same pace, which spreads
//    uneven work (sequences of different lengths, triangular key ranges).
//    Blocks past the last whole round of 8 chunks keep their index.
constexpr int kXcdChunk = 64;
__device__ __forceinline__ uint32_t xcd_remap(uint32_t i, uint32_t n, bool contiguous) {
  if (contiguous) {
    const uint32_t per = n / 8;
    return i < per * 8 ? (i % 8) * per + i / 8 : i;
  }
  const uint32_t span = 8 * kXcdChunk;
  if (i >= n / span * span) return i;
  const uint32_t k = i / 8;
  return ((i % 8) + 8 * (k / kXcdChunk)) * kXcdChunk + k % kXcdChunk;
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// The lanes of a wavefront exchange data through LDS here and there (each
// writes its own part, then reads what other lanes wrote).  The hardware runs
// a wave's LDS instructions in order, but the compiler knows nothing of the
// other lanes: without a fence it may move a read above another lane's write
// (into the branch that made that write conditional, say).  This orders every
// LDS access before it against every one after it, with all lanes present.
__device__ __forceinline__ void wave_lds_exchange() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

typedef int i32x4 __attribute__((ext_vector_type(4)));

// 16 bytes per lane from a buffer into LDS at byte address lds + 16*lane (LDS
// DMA; rsrc and lds are wave-uniform scalars).  Written as asm so that the
// compiler does not track the transfer: its wait-count pass would otherwise
// wait for every DMA in flight before any LDS read it cannot prove disjoint
// from the DMA's target (the V^T reads of the current tile, while the next
// tile's DMA is in flight).  The main loop waits for each tile's DMA itself
// (vmcnt) before the barrier that publishes the tile.  The host pass of the
// kernel templates sees empty bodies.
//
// The compiler inserts no wait states for an instruction inside asm, and the
// hardware does not interlock two of the operands here: a VMEM instruction
// that reads an SGPR written by a VALU instruction (v_readfirstlane, which
// builds the descriptors) needs 5 wait states, and an LDS DMA needs 1 after M0
// is written.  With fewer it can read the SGPR's previous value: a stale
// record count makes the fetch return zeros past it.  So the descriptors and
// the LDS base of a group of DMAs first pass through settle_sgprs (s_nop 4,
// which hands them back as its own outputs: every use comes after it, and
// only scalar arithmetic lies between), and each DMA then waits the one state
// M0 needs.

// A descriptor as read from the first lane (wave-uniform values in scalar
// registers: the compiler cannot hand an "s" asm operand a vector copy).
__device__ __forceinline__ i32x4 first_lane(i32x4 r) {
  return {__builtin_amdgcn_readfirstlane(r[0]), __builtin_amdgcn_readfirstlane(r[1]),
          __builtin_amdgcn_readfirstlane(r[2]), __builtin_amdgcn_readfirstlane(r[3])};
}
__device__ __forceinline__ void settle_sgprs(i32x4& r0, i32x4& r1, uint32_t& m) {
#if defined(__HIP_DEVICE_COMPILE__)
  r0 = first_lane(r0);
  r1 = first_lane(r1);
  m = (uint32_t)__builtin_amdgcn_readfirstlane((int)m);
  asm volatile("s_nop 4" : "+s"(r0), "+s"(r1), "+s"(m));
#endif
}
__device__ __forceinline__ void settle_sgprs(i32x4& r0, uint32_t& m) {
#if defined(__HIP_DEVICE_COMPILE__)
  r0 = first_lane(r0);
  m = (uint32_t)__builtin_amdgcn_readfirstlane((int)m);
  asm volatile("s_nop 4" : "+s"(r0), "+s"(m));
#endif
}
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t lds, int voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :: "v"(voff), "s"(rsrc), "{m0}"(lds) : "memory");
#endif
}

// ds_read_b64_tr_b16: inside each group of 16 lanes, lane i receives element
// k (k = 0..3) of the 8-byte row read by lane 4k + i/4, at position i%4.
__device__ __forceinline__ i16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (i16x4 __attribute__((address_space(3)))*)(p));
}

// Row index -> position of that row inside its sequence.  In the strided
// dense-row mode row r < nA is anchor r*gamma, later rows are tail rows.
template <int MODE>
__device__ __forceinline__ int row_pos(int r, int nA, int Lc, int gamma) {
  if (MODE == kDenseRows) return r < nA ? r * gamma : Lc + (r - nA);
  return r;
}

template <int D, int MODE>
__global__ __launch_bounds__(kAttnThreads) __attribute__((amdgpu_waves_per_eu(2)))
void attn_kernel(Args a) {
  using LD = Lds<D>;
  constexpr int NS = kAttnStages;
  // The sparse kernel also holds, after the K/V ring, the fp32 dense rows of
  // its block's anchors for the fused store: hpw * (slab rows / gamma) rows
  // of D floats, at most 128 * D floats (gamma >= 2).
  constexpr int kPreFloats = (MODE == kSparse) ? 128 * D : 0;
  __shared__ __attribute__((aligned(16))) uint16_t smem[NS * LD::stageElems + 2 * kPreFloats];
  float* const dpre = (float*)(smem + NS * LD::stageElems);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // The sparse kernel classifies tiles per wave from wave-uniform bounds:
  // with the wave index in a scalar register those tests stay scalar.
  const int wave = MODE == kSparse ? __builtin_amdgcn_readfirstlane(tid >> 6) : tid >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;

  // ---- which (sequence, head group, row tile[, key chunk]) this block owns
  // (grids hold fewer than 2^31 blocks; the divisors are the launch's)
  uint32_t lid = xcd_remap(blockIdx.x, gridDim.x, a.n_hgroups % 8 == 0);
  uint32_t q = fdiv(lid, a.fd_rtiles);
  int rt = (int)(lid - q * (uint32_t)a.n_rtiles);
  lid = q;
  int c = 0;
  if (MODE == kDenseRows) {
    q = fdiv(lid, a.fd_nC);
    c = (int)(lid - q * (uint32_t)a.nC);
    lid = q;
  }
  const int hg = (int)fdiv(lid, a.fd_B);
  const int b = (int)(lid - (uint32_t)hg * (uint32_t)a.B);
  // Longest rows first: in the dense modes blocks dispatched together then have
  // (nearly) the same number of key tiles, start on the same tile and stay in
  // step, so they share each key/value tile in L2.
  if (MODE == kDenseRows && a.dr_n1 > 0) {
    // Sequences of one length: every (row tile, chunk) pair that takes a whole
    // key chunk runs before any that takes part of one.  The whole-chunk
    // blocks all run the same number of tiles, so the blocks on one XCD stay
    // in step over a chunk's tiles from round to round of the dispatch (a
    // shorter diagonal block in between would start its CU on the next chunk
    // early and put it out of step with the others).
    int j = c * a.n_rtiles + rt;
    if (j < a.dr_n1) {
      c = 0;
      for (int f; c < a.nC - 1 && j >= (f = a.dr_nrt - a.dr_t[c]); ++c) j -= f;
      rt = a.dr_nrt - 1 - j;
    } else if ((j -= a.dr_n1) < a.dr_n2) {
      c = 0;
      for (int f; c < a.nC - 1 && j >= (f = a.dr_t[c] - a.dr_z[c]); ++c) j -= f;
      rt = a.dr_t[c] - 1 - j;
    } else {
      return;  // no key of any chunk is visible to this pair (uniform over the block)
    }
  } else if (MODE != kSparse) {
    rt = a.n_rtiles - 1 - rt;
  }

  const Seq sq = seq_of(a, b);
  const int L = sq.L;
  // hpw is a power of two: head in block = wave % hpw, sub-tile = wave / hpw
  const int hpw_log = __builtin_ctz(a.hpw);
  const int h = hg * a.hpw + (wave & (a.hpw - 1));
  const int g = (int)fdiv((uint32_t)(hg * a.hpw), a.fd_G);
  const int sub = wave >> hpw_log;
  const int nA = (int)fdiv((uint32_t)L, a.fd_gamma);
  const int Lc = nA * a.gamma;
  const int n_rows = (MODE == kDenseRows) ? nA + (L - Lc) : L;

  const int rows_per_block = kRowsPerWave * a.ppw;
  const int R0 = rt * rows_per_block;
  if (R0 >= n_rows) return;  // uniform over the block
  const int R1 = min(R0 + rows_per_block, n_rows);
  const int bpos_lo = row_pos<MODE>(R0, nA, Lc, a.gamma);
  const int bpos_hi = row_pos<MODE>(R1 - 1, nA, Lc, a.gamma);

  // ---- key tiles the block visits: [ta0, ta1) then [tb0, tb1)
  int ta0 = 0, ta1 = 0, tb0 = 0, tb1 = 0;
  // key-block lists: [ta0, ta1) indexes the block's list, then its own query
  // block's tiles [diag0, last row's tile]
  int lst0 = 0, diag0 = 0;
  if (MODE == kSparse && a.blk_ptr) {
    const int qb = (int)fdiv((uint32_t)R0, a.fd_bq);  // the block's rows lie in one query block
    const int64_t pi = ((int64_t)b * a.Hkv + g) * (a.nqb + 1) + qb;
    lst0 = a.blk_ptr[pi];
    ta1 = max(0, a.blk_ptr[pi + 1] - lst0);
    diag0 = qb * (a.block_q / kKeyTile);
    tb0 = diag0;
    tb1 = max(tb0, bpos_hi / kKeyTile + 1);
  } else if (MODE == kSparse) {
    const int sink_end = min(a.n_sink, bpos_hi + 1);
    ta1 = (sink_end + kKeyTile - 1) / kKeyTile;
    const int ws = max(0, bpos_lo - a.window + 1);
    tb0 = max(ws / kKeyTile, ta1);
    tb1 = max(tb0, bpos_hi / kKeyTile + 1);
  } else if (MODE == kDense) {
    ta1 = bpos_hi / kKeyTile + 1;
  } else {
    const int64_t kc0 = (int64_t)c * a.chunk;
    if (kc0 > bpos_hi) return;  // this key chunk lies past every row of the block
    const int64_t kc1 = min(kc0 + a.chunk, (int64_t)bpos_hi + 1);
    ta0 = (int)(kc0 / kKeyTile);
    ta1 = (int)((kc1 + kKeyTile - 1) / kKeyTile);
  }
  // The tile range is block-uniform; the list loads above are vector loads,
  // so say so explicitly, which keeps the loop counter and the per-tile tests
  // in scalar registers.
  ta0 = __builtin_amdgcn_readfirstlane(ta0);
  tb0 = __builtin_amdgcn_readfirstlane(tb0);
  lst0 = __builtin_amdgcn_readfirstlane(lst0);
  const int n_a = __builtin_amdgcn_readfirstlane(ta1 - ta0);
  const int n_iter = __builtin_amdgcn_readfirstlane(n_a + (tb1 - tb0));

  // ---- this wave's rows; lane (col) owns row wr0 + col
  const int wr0 = R0 + sub * kRowsPerWave;
  const bool wave_has_rows = wr0 < R1;
  const int my_r = wr0 + col;
  const bool row_valid = my_r < R1;
  const int my_pos = row_valid ? row_pos<MODE>(my_r, nA, Lc, a.gamma) : -1;
  const int wpos_lo = wave_has_rows ? row_pos<MODE>(wr0, nA, Lc, a.gamma) : 0;
  const int wpos_hi = wave_has_rows ? row_pos<MODE>(min(wr0 + kRowsPerWave, R1) - 1, nA, Lc,
                                                    a.gamma) : -1;

  bf16x8 qf[D / 16];  // the wave's queries (loaded in the prologue below)
  const int64_t kv_stride = (int64_t)a.Hkv * D;  // elements between consecutive keys
  const uint16_t* kbase = a.k + (sq.base * a.Hkv + g) * (int64_t)D;
  const uint16_t* vbase = a.v + (sq.base * a.Hkv + g) * (int64_t)D;

  // ---- tile loads by LDS DMA.  buffer_load_dwordx4 ... lds writes 16 bytes per
  // lane at M0 + 16*lane, so one instruction fills one 1 KB region of a tile.
  // Wave w fills regions w*RPW .. w*RPW+RPW-1 of both tiles; lane l of region
  // n lands on key row r = (1024n + 16l) / 2D at physical chunk pc and so
  // fetches logical chunk pc ^ swizzle(r) of that key.  The descriptors are
  // re-based at the tile's first key and end at the sequence end: keys past it
  // read as zero (and every valid row masks them).
  constexpr int RPW = LD::kRegionsPerWave;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  int dma_koff[RPW], dma_voff[RPW];
#pragma unroll
  for (int i = 0; i < RPW; ++i) {
    const int byte = (wave_s * RPW + i) * 1024 + 16 * lane;
    const int r = byte / (2 * D);
    const int pc = (byte % (2 * D)) / 16;
    dma_koff[i] = (int)(r * kv_stride * 2) + (pc ^ LD::kswz(r)) * 16;
    dma_voff[i] = (int)(r * kv_stride * 2) + (pc ^ LD::vswz(r)) * 16;
  }
  // Buffer descriptors (stride 0, raw buffer): base at the tile's first key,
  // num_records up to the sequence end, at most one tile.  Everything here is
  // wave-uniform (scalar registers).
  const uint32_t key_bytes = (uint32_t)__builtin_amdgcn_readfirstlane((int)(kv_stride * 2));
  const uint32_t tile_bytes = key_bytes * kKeyTile;
  const uint64_t kaddr0 = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uintptr_t)kbase) |
                          (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)((uintptr_t)kbase >> 32)) << 32;
  const uint64_t vaddr0 = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uintptr_t)vbase) |
                          (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)((uintptr_t)vbase >> 32)) << 32;
  const int L_s = __builtin_amdgcn_readfirstlane(L);
  const uint32_t smem_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint16_t*)smem;
  auto dma = [&](int tile, int stage) {
    if (tile < 0) return;  // a list entry the key set ignores
    const uint32_t tu = (uint32_t)__builtin_amdgcn_readfirstlane(tile);
    const uint64_t off = (uint64_t)tu * tile_bytes;
    int keys = L_s - (int)(tu * kKeyTile);
    keys = keys < 0 ? 0 : keys;
    keys = keys > kKeyTile ? kKeyTile : keys;
    const uint32_t nrec = (uint32_t)keys * key_bytes;
    const uint64_t ka = kaddr0 + off, va = vaddr0 + off;
    i32x4 kr = {(int)(uint32_t)ka, (int)((uint32_t)(ka >> 32) & 0xffffu), (int)nrec, 0x00020000};
    i32x4 vr = {(int)(uint32_t)va, (int)((uint32_t)(va >> 32) & 0xffffu), (int)nrec, 0x00020000};
    uint32_t st0 = smem_lds + (uint32_t)(stage * LD::stageElems) * 2;
    settle_sgprs(kr, vr, st0);
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
      const uint32_t region = (uint32_t)((wave_s * RPW + i) * 512) * 2;  // bytes
      dma16(kr, st0 + region, dma_koff[i]);
      dma16(vr, st0 + (uint32_t)LD::kElems * 2 + region, dma_voff[i]);
    }
  };

  // Per-lane LDS read offsets (elements, stage 0).  K operand (nb, kk): key row
  // 32nb + col, logical chunk 2kk + half.  V^T operand (t, mb): transposing
  // reads where, inside each 16-lane group, lane 4k+m points at key
  // 16t + 4h + k (and +8 for the second read) and dims 32mb + 16*g1 + 4m.
  const int ksw = LD::kswz(col);
  int kread[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) kread[kk] = col * D + (((2 * kk + half) ^ ksw) * 8);
  const int tr_g1 = (lane >> 4) & 1, tr_k = (lane >> 2) & 3, tr_m = lane & 3;
  const int vsw = LD::vswz(4 * half + tr_k);
  int vread[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
    vread[mb] = (4 * half + tr_k) * D + (((4 * mb + 2 * tr_g1 + (tr_m >> 1)) ^ vsw) * 8) +
                (tr_m & 1) * 4;

  // list entries outside [0, diag0) are not part of the key set (-1: skipped)
  auto tile_at = [&](int it) -> int {
    if (it >= n_a) return tb0 + (it - n_a);
    if (MODE == kSparse && a.blk_ptr) {
      const int e = __builtin_amdgcn_readfirstlane(a.blk_idx[lst0 + it]);
      return (e >= 0 && e < diag0) ? e : -1;
    }
    return ta0 + it;
  };

  // 0: no key of the tile is visible to any row of the wave; 1: every key is
  // visible to every row; otherwise the mask the tile needs per element:
  // kMaskCausal (some key lies past some row), kMaskWindow (some key lies
  // before some row's window), kMaskBoth, or kMaskAll (the window test meets
  // sink keys).  The dense modes only ever need the causal mask.
  auto classify = [&](int tile) -> int {
    if (!wave_has_rows || tile < 0) return 0;
    const int k0 = tile * kKeyTile, k1 = k0 + kKeyTile - 1;
    if (k0 > wpos_hi) return 0;
    if (MODE == kSparse) {
      if (k0 >= a.n_sink && wpos_lo - k1 >= a.window) return 0;
      const bool need_c = k1 > wpos_lo;
      const bool need_w = k1 >= a.n_sink && (int64_t)wpos_hi - k0 >= a.window;
      if (need_w && k0 < a.n_sink) return kMaskAll;
      return need_c ? (need_w ? kMaskBoth : kMaskCausal) : (need_w ? kMaskWindow : 1);
    }
    return k1 <= wpos_lo ? 1 : kMaskCausal;
  };

  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};
  // Reference `ref` of the base-2 logits (same in lanes l and l^32; has_ref: a
  // reference exists) and -ref / c in every register of nref, the block the
  // score accumulators start from, so that c times them is logit - ref.
  // (Scaling the queries by c ahead of the MFMA would round c q to bf16 once
  // more, an error proportional to the logits themselves.)
  const float qscale = a.scale_log2, inv_qscale = 1.f / a.scale_log2;
  float ref = 0.f;
  bool has_ref = false;
  f32x16 nref = f32x16{};
  float l = 0.f;        // this lane's share of the softmax normaliser
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  // S^T of one tile against the wave's rows (register r of lane half h holds
  // key 8*(r/4) + 4*h + r%4 in s0, that key + 32 in s1); keys outside a row's
  // key set read -inf when `masked`.
  auto qk = [&](const uint16_t* ks, int tile, int masked, f32x16& s0, f32x16& s1) {
    s0 = nref;
    s1 = nref;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      const bf16x8 ka = *(const bf16x8*)(ks + kread[kk]);
      const bf16x8 kb = *(const bf16x8*)(ks + kread[kk] + 32 * D);
      s0 = mfma32(ka, qf[kk], s0);
      s1 = mfma32(kb, qf[kk], s1);
    }
    // issue the K reads four MFMAs ahead of their use, so the matrix phase is
    // not paced by LDS latency
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int i = 0; i < D / 8 - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    // accumulator register r of lane half h holds key kbase_t + o with the
    // constant offset o = 8*(r/4) + r%4 (+32 in s1); the tests compare o
    // against per-lane bounds: causal o <= my_pos - kbase_t, window
    // o > my_pos - kbase_t - window, sink o < n_sink - kbase_t
    if (masked) {
      const int kbase_t = tile * kKeyTile + 4 * half;
      const int lim_c = my_pos - kbase_t;
      // (64-bit: the window may be as large as INT_MAX; every offset is >= 0,
      // so a bound clamped at -1 admits the whole tile, as such a window does)
      const int lim_w = (int)max((int64_t)lim_c - (int64_t)a.window, (int64_t)-1);
      const int lim_s = a.n_sink - kbase_t;
      // one element test per mask kind (the kind is wave-uniform in the sparse
      // mode, so each is a branch of its own)
      auto apply = [&](auto ok) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int o0 = 8 * (r >> 2) + (r & 3);
          s0[r] = ok(o0) ? s0[r] : -INFINITY;
          s1[r] = ok(o0 + 32) ? s1[r] : -INFINITY;
        }
      };
      if (MODE != kSparse || masked == kMaskCausal)
        apply([&](int o) { return o <= lim_c; });
      else if (masked == kMaskWindow)
        apply([&](int o) { return o > lim_w; });
      else if (masked == kMaskBoth)
        apply([&](int o) { return o <= lim_c && o > lim_w; });
      else
        apply([&](int o) { return o <= lim_c && (o < lim_s || o > lim_w); });
    }
  };

  // Online-softmax update with one tile's scores: the accumulators hold
  // s = q.k - ref / c, so c s = logit - ref in base-2 units, with c =
  // log2(e)/sqrt(d) applied in fp32 here (the queries stay as given); adds
  // the tile's weights to l and returns them as bf16 P^T fragments, moving
  // the reference first when it has to.
  //
  // The reference lags the true running max: weights are taken against the
  // current one, and only if some lane's share of the tile's weight sum exceeds
  // 2^13 (or some lane has no reference yet) does the wave take the row max
  // of the tile.  ref then moves up by it when a score exceeds ref by more than 8
  // (a weight above 2^8), rescaling O and l, and the weights are taken again.
  // Every weight stays below 2^13 (harmless in fp32 and bf16): a lane whose
  // scores all lie within 8 of ref sums at most 32 * 2^8 = 2^13.  The result is
  // the same either way, since numerator and normaliser share the reference;
  // the common tile pays no max reduction and no subtraction.
  auto softmax = [&](f32x16& s0, f32x16& s1, bf16x8* pf) {
    // P^T fragment t covers keys 16t..16t+15: registers 8*(t%2)..+7 of block
    // t/2.  The sum covers the bf16 weights the MFMA multiplies (dot2 with 1,1),
    // in two chains.
    auto weights = [&]() {
      f32x16 p0, p1;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        p0[i] = fast_exp2(qscale * s0[i]);
        p1[i] = fast_exp2(qscale * s1[i]);
      }
      pf[0] = __builtin_convertvector(p0.lo, bf16x8);
      pf[1] = __builtin_convertvector(p0.hi, bf16x8);
      pf[2] = __builtin_convertvector(p1.lo, bf16x8);
      pf[3] = __builtin_convertvector(p1.hi, bf16x8);
      float ta = 0.f, tb = 0.f;
#pragma unroll
      for (int f = 0; f < 4; ++f) {
        ta = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[f], pf[f], 0, 1), ones2, ta, false);
        tb = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[f], pf[f], 2, 3), ones2, tb, false);
        ta = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[f], pf[f], 4, 5), ones2, ta, false);
        tb = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pf[f], pf[f], 6, 7), ones2, tb, false);
      }
      // the exponentials go two at a time with other VALU instructions (the
      // scaling multiplies, conversions, sums) between them: a wave issues one
      // exponential every ~15 clocks and fits its other VALU work into those
      // gaps
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x400, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
      }
      return ta + tb;
    };
    float t = INFINITY;
    if (!__any(!has_ref)) t = weights();
    if (__any(!(t <= 8192.f))) {
      // row max over the 32 scores of this lane (a tree of 3-input max), then
      // across the lane pair l, l^32 that shares the row
      float t3[11];
#pragma unroll
      for (int i = 0; i < 5; ++i) t3[i] = fmaxf(s0[3 * i], fmaxf(s0[3 * i + 1], s0[3 * i + 2]));
#pragma unroll
      for (int i = 0; i < 5; ++i) t3[5 + i] = fmaxf(s1[3 * i], fmaxf(s1[3 * i + 1], s1[3 * i + 2]));
      t3[10] = fmaxf(s0[15], s1[15]);
      float mx = fmaxf(fmaxf(fmaxf(t3[0], t3[1]), fmaxf(t3[2], t3[3])),
                       fmaxf(fmaxf(t3[4], t3[5]), fmaxf(t3[6], t3[7])));
      mx = fmaxf(mx, fmaxf(t3[8], fmaxf(t3[9], t3[10])));
      {
        const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                         false, false);
        mx = qscale * fmaxf(__uint_as_float(pr[0]), __uint_as_float(pr[1]));  // base 2
      }
      // a lane without a reference takes its tile max (if it sees any key);
      // one with a reference moves only up
      const bool seen = mx != -INFINITY;
      const bool grow = has_ref ? mx > 8.f : seen;
      if (__any(grow)) {
        const float dm = has_ref ? fmaxf(mx, 0.f) : (seen ? mx : 0.f);
        const float alpha = has_ref ? fast_exp2(-dm) : 0.f;  // l and O are still zero without one
        ref += dm;
        has_ref = has_ref || seen;
        l *= alpha;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
        const float dr = dm * inv_qscale;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          s0[i] -= dr;
          s1[i] -= dr;
          nref[i] = -ref * inv_qscale;
        }
      }
      t = weights();
    }
    l += t;
  };

  // O^T += V^T P^T for one tile.
  auto pv = [&](const uint16_t* vs, const bf16x8* pf) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) {
        const i16x4 lo = lds_read_tr(vs + vread[mb] + (16 * t) * D);
        const i16x4 hi = lds_read_tr(vs + vread[mb] + (16 * t + 8) * D);
        const i16x8 both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[mb] = mfma32(__builtin_bit_cast(bf16x8, both), pf[t], o[mb]);
      }
    }
    // V^T reads (two per MFMA) four MFMAs ahead of their use
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int i = 0; i < D / 8 - 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  };

  auto compute = [&](const uint16_t* ks, int tile, int masked) {
    f32x16 s0, s1;
    bf16x8 pf[4];
    qk(ks, tile, masked, s0, s1);
    softmax(s0, s1, pf);
    pv(ks + LD::kElems, pf);
  };

  // ---- prologue: the first tile's DMA, the queries and the staged dense rows
  // are all in flight before the block waits once for them.
  //
  // A stage holds the tile of its last DMA; lanes past the sequence end are
  // written as zeros.  Only a block whose first NS tiles include its last one
  // (the only tile that can end inside the sequence's last 64 keys) clears
  // the ring first, so that no stage can hold bits left by an earlier kernel.
  if (n_iter <= NS) {
    for (int i = tid; i < NS * LD::stageElems / 8; i += kAttnThreads)
      *(u32x4*)(smem + 8 * i) = u32x4{0u, 0u, 0u, 0u};
    __syncthreads();
  }
#pragma unroll
  for (int p = 0; p < NS - 1; ++p)
    if (p < n_iter) dma(tile_at(p), p);

  // Fused store: the merged dense rows of the block's anchors whose Delta is
  // not zero (anchor slot = head in block * groups per slab + group in slab),
  // staged in LDS so the epilogue does not wait on memory.  Each thread's
  // first vector loads with the queries; gamma < 16 (d = 128) leaves more.
  const bool stage_dense = MODE == kSparse && a.fuse && a.gamma > 1;
  const int per_slab = (int)fdiv((uint32_t)(kRowsPerWave * a.ppw), a.fd_gamma);
  const int nvec = stage_dense ? a.hpw * per_slab * (D / 4) : 0;
  auto dense_src = [&](int u) -> const f32x4* {
    const int slot = u / (D / 4), dv = u % (D / 4);
    const int apos = R0 + (slot % per_slab) * a.gamma;
    if (apos >= min(R1, Lc) || (int64_t)apos < a.cover) return nullptr;
    const int hh = hg * a.hpw + slot / per_slab;
    return (const f32x4*)(a.dense + (((int64_t)b * a.Hq + hh) * a.nR_max +
                                     (int)fdiv((uint32_t)apos, a.fd_gamma)) * D + dv * 4);
  };

  // Q fragments: lane holds dims kk*16 + half*8 .. +8 of its row, for every kk.
  // Rows past the end of the block load row R1-1's query (a valid row) and are
  // never written, so no load sits behind a branch.
  //
  // The sparse kernel, whose blocks are short, fetches its queries by LDS DMA
  // instead: whole rows (four per instruction at d = 128), each lane fetching
  // the 16-byte chunk that lands, XOR-swizzled by row, at its place in LDS.
  // The staging is free LDS: ring stage 1 (filled only after the first
  // barrier) for waves 0-3, the upper half of the dense-row area for waves
  // 4-7 (when the staged dense rows fit the lower half).  Each lane reads its
  // fragments from there.  Read straight into the fragment layout, every load
  // instruction fetched 32 bytes of each of 32 rows, and at every block's start
  // those loads queued behind each other in the memory pipeline.
  constexpr int QCPR = D / 8;  // 16-byte chunks per query row
  const bool q_lds = MODE == kSparse && nvec * 4 <= 64 * D;
  uint16_t* const qst = smem + (wave < 4 ? LD::stageElems + wave * (kRowsPerWave * D)
                                         : NS * LD::stageElems + 128 * D + (wave - 4) * (kRowsPerWave * D));
  if (q_lds) {
    static_assert(NS == 2 && 4 * kRowsPerWave * D <= LD::stageElems, "query staging fits stage 1");
    constexpr int RPI = 64 / QCPR;  // rows per DMA instruction
    const int jl = lane / QCPR, pc = lane % QCPR;
    const uint32_t row_bytes = (uint32_t)__builtin_amdgcn_readfirstlane(a.Hq * D * 2);
    const uint16_t* q0 = a.q + ((sq.base + R0) * a.Hq + h) * (int64_t)D;
    const uint64_t qa = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uintptr_t)q0) |
                        (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)((uintptr_t)q0 >> 32)) << 32;
    i32x4 qr = {(int)(uint32_t)qa, (int)((uint32_t)(qa >> 32) & 0xffffu), (int)0xfffffff0u, 0x00020000};
    uint32_t qdst = smem_lds + (uint32_t)(qst - smem) * 2;
    settle_sgprs(qr, qdst);
#pragma unroll
    for (int i = 0; i < kRowsPerWave / RPI; ++i) {
      const int j = i * RPI + jl;  // row of the wave
      const int r = min(wr0 + j, R1 - 1);
      dma16(qr, qdst + i * 1024, (r - R0) * (int)row_bytes + ((pc ^ (j & (QCPR - 1))) * 16));
    }
  } else {
    const int pos_ld = row_valid ? my_pos : row_pos<MODE>(R1 - 1, nA, Lc, a.gamma);
    const uint16_t* qp = a.q + ((sq.base + pos_ld) * a.Hq + h) * (int64_t)D + half * 8;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *(const bf16x8*)(qp + kk * 16);
  }
  const f32x4* dsrc = tid < nvec ? dense_src(tid) : nullptr;
  f32x4 dreg = f32x4{};
  if (dsrc) dreg = *dsrc;
  // Everything above has landed after this wait (vmcnt(0)): the main loop's
  // MFMAs read qf every iteration and must not wait behind the DMA issued in
  // it, and the first tile is in this wave's part of stage 0.
  __builtin_amdgcn_s_waitcnt(0x0F70);
  if (q_lds) {
    // this wave's query rows have landed in its staging (each lane reads
    // chunks other lanes fetched)
    wave_lds_exchange();
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk)
      qf[kk] = *(const bf16x8*)(qst + col * D + (((2 * kk + half) ^ (col & (QCPR - 1))) * 8));
    // the fragments are in registers before the barrier after which stage 1 fills
    __builtin_amdgcn_s_waitcnt(0xC07F);
  }
  if (dsrc) *(f32x4*)(dpre + tid * 4) = dreg;
  for (int u = tid + kAttnThreads; u < nvec; u += kAttnThreads)
    if (const f32x4* src = dense_src(u)) *(f32x4*)(dpre + u * 4) = *src;

  // ---- main loop over a ring of NS LDS stages, one barrier per tile.  Step
  // `it` waits until this wave's DMA of tile it has landed (later tiles may
  // still be in flight), meets the other waves at the barrier (after which
  // tile it is in LDS for everyone and nobody reads stage (it-1) % NS any
  // more), starts the DMA of tile it+NS-1 into that stage, then computes
  // tile it.  Keys past the sequence end arrive as zeros from the DMA; a
  // stage is read only after a DMA has filled it.
  constexpr int kLoadsPerTile = 2 * RPW;  // vmcnt entries one tile's DMA adds per wave
  // The loop is unrolled by the ring depth so each step's stage is a constant:
  // the LDS operand addresses are then a loop-invariant per-lane register plus
  // an immediate offset, with no address arithmetic per tile.
  for (int it0 = 0; it0 < n_iter; it0 += NS) {
#pragma unroll
    for (int st = 0; st < NS; ++st) {
      const int it = it0 + st;
      if (it >= n_iter) break;
      const int ahead = min(NS - 2, n_iter - 1 - it);  // later tiles already in flight
      if (NS >= 4 && ahead >= 2)
        __builtin_amdgcn_s_waitcnt(0x0F70 | ((2 * kLoadsPerTile) & 15) | (((2 * kLoadsPerTile) >> 4) << 14));
      else if (NS >= 3 && ahead >= 1)
        __builtin_amdgcn_s_waitcnt(0x0F70 | (kLoadsPerTile & 15) | ((kLoadsPerTile >> 4) << 14));
      else
        __builtin_amdgcn_s_waitcnt(0x0F70);
      __syncthreads();
      if (it + NS - 1 < n_iter) dma(tile_at(it + NS - 1), (st + NS - 1) % NS);
      const int tile = tile_at(it);
      const int cls = classify(tile);
      const uint16_t* ks = smem + st * LD::stageElems;
      if (MODE == kSparse) {
        // tile classes are scalar here: one copy of the tile body with the
        // mask as a branch inside it, so the accumulators keep one register
        // assignment across tiles (two copies made the compiler copy O
        // between them at every step)
        if (cls != 0) compute(ks, tile, cls == 1 ? 0 : cls);
      } else if (cls == 1) {
        compute(ks, tile, 0);
      } else if (cls != 0) {
        compute(ks, tile, kMaskCausal);
      }
    }
  }

  // ---- epilogue: output register r of block mb is dim 32*mb + 8*(r/4) + 4*half + r%4
  const float lt = l + __shfl_xor(l, 32);
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  if (MODE == kSparse) {
    const float inv = 1.f / lt;
    f32x4 val[D / 32][4];  // this lane's output row in fp32
    if (a.fuse) {
      // Fused Delta store (the dense rows were merged into a.dense beforehand).
      // Every group of gamma rows lies inside one head's row slab of this
      // block, so its anchor's sparse row is in a register of some lane here:
      // the anchor lane forms Delta = dense - sparse in fp32 over the dense row
      // the prologue staged in LDS and leaves it there for the group's other
      // rows, which store bf16(sparse + Delta), one rounding.  Anchor rows
      // store the dense row, tail rows (past the last whole group) the dense
      // row too; groups whose anchor lies below a.cover (a < n_sink + window:
      // its sparse key set is all of [0, a]) have Delta = 0 exactly and keep
      // the sparse row untouched.  Recompute (fuse 2) replaces anchors only.
      const bool in_c = row_valid && my_pos < Lc;
      // group of the row inside the block's slab (R0 is a multiple of gamma)
      const int grp = in_c ? (int)fdiv((uint32_t)(my_pos - R0), a.fd_gamma) : 0;
      const int anc = in_c ? R0 + grp * a.gamma : 0;
      const bool open = in_c && (int64_t)anc >= a.cover;
      const bool is_anchor = open && anc == my_pos;
      const bool staged = a.gamma > 1;  // anchor dense rows are in dpre
      const bool delta = a.fuse == 1 && staged;
      const int xslot = ((wave & (a.hpw - 1)) * per_slab + grp) * D;
      if (delta && is_anchor) {
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq) {
            const int dim = 32 * mb + 8 * jq + 4 * half;
            const f32x4 sv = {o[mb][4 * jq] * inv, o[mb][4 * jq + 1] * inv,
                              o[mb][4 * jq + 2] * inv, o[mb][4 * jq + 3] * inv};
            const f32x4 dv = *(const f32x4*)(dpre + xslot + dim);
            *(f32x4*)(dpre + xslot + dim) = dv - sv;
            val[mb][jq] = dv;
          }
      }
      // Delta of every group is in dpre, and no wave reads the K/V ring any more
      __syncthreads();
      const bool tail = row_valid && my_pos >= Lc;
      // one branch per row kind (not one per vector): corrected rows fold the
      // normalisation into the add, sparse rows only normalise, dense rows copy
      if (delta && is_anchor) {
        // val holds the dense row
      } else if (delta && open) {
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq) {
            const f32x4 dl = *(const f32x4*)(dpre + xslot + 32 * mb + 8 * jq + 4 * half);
#pragma unroll
            for (int e = 0; e < 4; ++e) val[mb][jq][e] = __builtin_fmaf(o[mb][4 * jq + e], inv, dl[e]);
          }
      } else if (tail || (is_anchor && !staged)) {
        // dense row in global memory: tail rows, and anchors when not staged
        const float* gdrow =
            a.dense + (((int64_t)b * a.Hq + h) * a.nR_max +
                       (in_c ? (int)fdiv((uint32_t)my_pos, a.fd_gamma) : nA + (my_pos - Lc))) * D;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq) val[mb][jq] = *(const f32x4*)(gdrow + 32 * mb + 8 * jq + 4 * half);
      } else if (is_anchor) {
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq)
            val[mb][jq] = *(const f32x4*)(dpre + xslot + 32 * mb + 8 * jq + 4 * half);
      } else {
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq)
#pragma unroll
            for (int e = 0; e < 4; ++e) val[mb][jq][e] = o[mb][4 * jq + e] * inv;
      }
    } else {
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq)
#pragma unroll
          for (int e = 0; e < 4; ++e) val[mb][jq][e] = o[mb][4 * jq + e] * inv;
      // the unfused schedule also keeps every anchor's sparse row in fp32
      const int grp = (a.sa && row_valid) ? (int)fdiv((uint32_t)my_pos, a.fd_gamma) : 0;
      if (a.sa && row_valid && grp * a.gamma == my_pos && my_pos < Lc) {
        float* sarow = a.sa + (((int64_t)b * a.Hq + h) * a.nA_max + grp) * D;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq) *(f32x4*)(sarow + 32 * mb + 8 * jq + 4 * half) = val[mb][jq];
      }
      __syncthreads();  // no wave reads the K/V ring any more
    }
    // The rows go out through LDS: each lane writes its row as bf16 into its
    // wave's 32 x D region of the idle K/V ring (16-byte chunks XOR-swizzled
    // by row), then every store instruction writes whole rows (64 lanes x 16
    // bytes: four rows at d = 128) instead of 16 bytes of each of 32 rows
    // that lie Hq * d elements apart.  The wave reads only what it wrote (its
    // lanes exchange rows through wave_lds_exchange).
    static_assert(NS * LD::stageElems >= kAttnWaves * kRowsPerWave * D, "output staging fits the ring");
    constexpr int CPR = D / 8;     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;  // rows per store instruction
    uint16_t* const stg = smem + wave * (kRowsPerWave * D);
    if (row_valid) {
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq)
          *(bf16x4*)(stg + col * D + (((4 * mb + jq) ^ (col & (CPR - 1))) * 8) + 4 * half) =
              __builtin_convertvector(val[mb][jq], bf16x4);
    }
    wave_lds_exchange();
    // All the wave's reads first (one wait for them), then the stores: row
    // wr0 + rr of the wave lies rr * Hq * D elements past row wr0.
    const int rsub = lane / CPR, cc = lane % CPR;
    constexpr int NI = kRowsPerWave / RPI;
    u32x4 w[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int rr = i * RPI + rsub;
      w[i] = *(const u32x4*)(stg + rr * D + ((cc ^ (rr & (CPR - 1))) * 8));
    }
    uint16_t* const orow = a.out + ((sq.base + wr0 + rsub) * a.Hq + h) * (int64_t)D + cc * 8;
    const int64_t rstep = (int64_t)RPI * a.Hq * D;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (wr0 + i * RPI + rsub < R1) *(u32x4*)(orow + i * rstep) = w[i];
    return;
  }
  if (MODE == kDenseRows) {
    // Unnormalised partial rows of this key chunk, through the idle ring like
    // the sparse rows: each lane writes its fp32 row into its wave's 16 x D
    // region (16-byte chunks XOR-swizzled by row), two passes of 16 rows, so
    // that every store instruction writes whole rows (two of 512 bytes at
    // d = 128) instead of 32 bytes of each of 32 rows nC * D floats apart.
    __syncthreads();  // no wave reads the K/V ring any more
    static_assert(NS * LD::stageElems * 2 >= kAttnWaves * 16 * D * 4, "partial staging fits the ring");
    constexpr int CPR = D / 4;     // 16-byte chunks per fp32 row
    constexpr int RPI = 64 / CPR;  // rows per store instruction
    float* const stg = (float*)smem + wave * (16 * D);
    const int rsub = lane / CPR, cc = lane % CPR;
    const int64_t row0 = ((int64_t)b * a.Hq + h) * a.nR_max;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
      if (pass) wave_lds_exchange();  // the first pass's reads are done
      if (row_valid && (col >> 4) == pass) {
        const int r16 = col & 15;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
          for (int jq = 0; jq < 4; ++jq)
            *(f32x4*)(stg + r16 * D + (((8 * mb + 2 * jq + half) ^ (r16 & (CPR - 1))) * 4)) =
                f32x4{o[mb][4 * jq], o[mb][4 * jq + 1], o[mb][4 * jq + 2], o[mb][4 * jq + 3]};
      }
      wave_lds_exchange();
      // reads first, then the stores (row r lies r * nC * D floats past row 0)
      constexpr int NI = 16 / RPI;
      f32x4 w[NI];
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int rr = i * RPI + rsub;
        w[i] = *(const f32x4*)(stg + rr * D + ((cc ^ (rr & (CPR - 1))) * 4));
      }
      const int rb = wr0 + 16 * pass + rsub;
      float* const prow = a.part_o + ((row0 + rb) * a.nC + c) * D + cc * 4;
      const int64_t rstep = (int64_t)RPI * a.nC * D;
#pragma unroll
      for (int i = 0; i < NI; ++i)
        if (rb + i * RPI < R1) *(f32x4*)(prow + i * rstep) = w[i];
    }
    if (row_valid && half == 0) {
      const int64_t slot = (row0 + my_r) * a.nC + c;
      a.part_ml[slot * 2] = has_ref ? ref : -INFINITY;  // -inf when no key of the chunk is visible
      a.part_ml[slot * 2 + 1] = lt;
    }
    return;
  }
  if (!row_valid) return;
  const float inv = 1.f / lt;
  uint16_t* orow = a.out + ((sq.base + my_pos) * a.Hq + h) * (int64_t)D;
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) {
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const int dim = 32 * mb + 8 * jq + 4 * half;
      f32x4 val = {o[mb][4 * jq] * inv, o[mb][4 * jq + 1] * inv, o[mb][4 * jq + 2] * inv,
                   o[mb][4 * jq + 3] * inv};
      *(bf16x4*)(orow + dim) = __builtin_convertvector(val, bf16x4);
    }
  }
}

// Step 3 of Algorithm 1 for one dense row r of one sequence and a range of
// heads: merge the key-chunk partials of r into the dense result (log-sum-exp
// merge), then
//   anchor row a = r*gamma:  Delta = dense - sparse(a) in fp32, out[a] = dense,
//                            out[i] += Delta for i = a+1 .. a+gamma-1;
//   tail row:                out[row] = dense.
// An anchor below a.cover (a < n_sink + window: all keys 0..a are in its
// sparse set) has Delta exactly zero and the block leaves its rows untouched;
// with key-block lists no anchor is assumed covered (cover = 0).
// Epilogue modes: the Delta correction itself; "recompute" (Eq. 5: the dense
// row replaces the sparse one at anchors only); merge only (Delta_i into
// dbuf for the other correction variants, tail rows into out); or, for the
// fused schedule, which runs before the sparse kernel, the merged dense rows
// into a.dense in fp32 (covered anchors are skipped: their groups keep the
// sparse rows).
enum Epi { kEpiDelta = 0, kEpiRecompute = 1, kEpiMergeOnly = 2, kEpiMergeDense = 3 };

template <int D, int EPI>
__global__ __launch_bounds__(kEpiThreads) void delta_epilogue_kernel(Args a) {
  __shared__ float delta[8192];  // [head in range][D]
  const int tid = threadIdx.x;
  int64_t lid = blockIdx.x;
  const int n_hc = (a.Hq + a.head_chunk - 1) / a.head_chunk;
  const int hc = (int)(lid % n_hc);
  lid /= n_hc;
  const int r = (int)(lid % a.nR_max);
  const int b = (int)(lid / a.nR_max);

  const Seq sq = seq_of(a, b);
  const int L = sq.L;
  const int nA = L / a.gamma;
  const int Lc = nA * a.gamma;
  const int nR = nA + (L - Lc);
  if (r >= nR) return;
  const bool anchor = r < nA;
  const int pos = anchor ? r * a.gamma : Lc + (r - nA);
  const bool covered = anchor && (int64_t)pos < a.cover;
  const int h0 = hc * a.head_chunk;
  const int h1 = min(a.Hq, h0 + a.head_chunk);
  const int nh = h1 - h0;
  constexpr int DC = D / 8;
  if (covered) {
    if (EPI == kEpiMergeOnly) {  // Delta_i is exactly zero
      for (int idx = tid; idx < nh * DC; idx += kEpiThreads) {
        const int h = h0 + idx / DC, dc = idx % DC;
        *(f32x8*)(a.dbuf + (((int64_t)b * a.Hq + h) * a.nA_max + r) * D + dc * 8) = f32x8{};
      }
    }
    return;
  }
  const int nc = (int)(((int64_t)pos + a.chunk) / a.chunk);  // chunks holding keys 0..pos
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

  for (int idx = tid; idx < nh * DC; idx += kEpiThreads) {
    const int hh = idx / DC, dc = idx % DC;
    const int h = h0 + hh;
    const int64_t slot0 = (((int64_t)b * a.Hq + h) * a.nR_max + r) * a.nC;
    // one pass with a running max M (the loads of every chunk are independent,
    // so they can all be in flight together): chunks with no visible key
    // (max -inf) are skipped, and acc, lsum move to a larger M by 2^(M - Mn)
    float M = -INFINITY, lsum = 0.f;
    f32x8 acc = f32x8{};
#pragma unroll 4
    for (int cc = 0; cc < nc; ++cc) {
      const float mc = a.part_ml[(slot0 + cc) * 2];
      const float lc = a.part_ml[(slot0 + cc) * 2 + 1];
      const f32x8 po = *(const f32x8*)(a.part_o + (slot0 + cc) * D + dc * 8);
      if (mc == -INFINITY) continue;
      const float Mn = fmaxf(M, mc);
      const float sc = fast_exp2(M - Mn), w = fast_exp2(mc - Mn);
      lsum = lsum * sc + w * lc;
      acc = acc * sc + w * po;
      M = Mn;
    }
    const f32x8 dense = acc * (1.f / lsum);
    if (EPI == kEpiMergeDense) {
      *(f32x8*)(a.dense + (((int64_t)b * a.Hq + h) * a.nR_max + r) * D + dc * 8) = dense;
      continue;
    }
    uint16_t* orow = a.out + ((sq.base + pos) * a.Hq + h) * (int64_t)D + dc * 8;
    if (EPI != kEpiMergeOnly || !anchor) *(bf16x8_t*)orow = __builtin_convertvector(dense, bf16x8_t);
    if (anchor && EPI != kEpiRecompute) {
      const int64_t arow = (((int64_t)b * a.Hq + h) * a.nA_max + r) * D + dc * 8;
      const f32x8 dl = dense - *(const f32x8*)(a.sa + arow);
      if (EPI == kEpiDelta)
        *(f32x8*)(delta + hh * D + dc * 8) = dl;
      else
        *(f32x8*)(a.dbuf + arow) = dl;
    }
  }
  if (!anchor || EPI != kEpiDelta) return;
  __syncthreads();

  // rows pos+1 .. pos+gamma-1 for heads [h0, h1): nh*D contiguous values per
  // row.  Each thread loads kU vectors before it stores any, so that many
  // reads per thread are in flight (a load and a store of one address per
  // iteration would leave one).
  constexpr int kU = 4;
  const int per_row = nh * DC;
  const int64_t total = (int64_t)(a.gamma - 1) * per_row;
  for (int64_t u0 = tid; u0 < total; u0 += (int64_t)kU * kEpiThreads) {
    uint16_t* p[kU];
    bf16x8_t x[kU];
    int dl[kU];
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      const int64_t u = min(u0 + (int64_t)j * kEpiThreads, total - 1);
      const int i = (int)(u / per_row);
      const int rem = (int)(u % per_row);
      const int hh = rem / DC, dc = rem % DC;
      p[j] = a.out + ((sq.base + pos + 1 + i) * a.Hq + h0 + hh) * (int64_t)D + dc * 8;
      dl[j] = hh * D + dc * 8;
      x[j] = *(const bf16x8_t*)p[j];
    }
#pragma unroll
    for (int j = 0; j < kU; ++j) {
      if (u0 + (int64_t)j * kEpiThreads >= total) break;
      const f32x8 y = __builtin_convertvector(x[j], f32x8) + *(const f32x8*)(delta + dl[j]);
      *(bf16x8_t*)p[j] = __builtin_convertvector(y, bf16x8_t);
    }
  }
}

// Recurrences of the smoothing variants over the anchors of one sequence,
// one thread per (sequence, head, channel), in anchor order (a group's state
// needs the previous group's):
//   EMA (weight w): E_r = (1-w) E_{r-1} + w D_r over D = repeat(Delta, gamma),
//     E_{-1} = D_0.  Inside group i, D is constant, so with q = 1-w the value
//     entering the group, Ein_i, gives E_{a_i+k} = q^(k+1) Ein_i +
//     (1 - q^(k+1)) Delta_i; the scan stores Ein_i and steps
//     Ein_{i+1} = q^gamma Ein_i + (1 - q^gamma) Delta_i.
//   alpha-beta-gamma filter (gain p0, p1, p2; the interpolation appendix's
//     filter algorithm): a linear state-space recursion over the anchors;
//     Delta_i is replaced by the filtered position.
template <int CORR>
__global__ __launch_bounds__(256) void corr_scan_kernel(Args a) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_seq = (int64_t)a.Hq * a.d;
  if (t >= (int64_t)a.B * per_seq) return;
  const int b = (int)(t / per_seq);
  const int h = (int)((t % per_seq) / a.d);
  const int c = (int)(t % a.d);
  const int nA = seq_of(a, b).L / a.gamma;
  if (nA == 0) return;
  float* dl = a.dbuf + ((int64_t)b * a.Hq + h) * a.nA_max * a.d + c;
  // anchors are visited in batches of kB whose loads are all issued before the
  // recurrence consumes them, so the scan is not bound by one load at a time
  constexpr int kB = 16;
  float buf[kB];
  if (CORR == 3) {
    float* ein = a.ebuf + ((int64_t)b * a.Hq + h) * a.nA_max * a.d + c;
    const float q = 1.f - a.corr_p[0];
    const float qg = (q == 0.f) ? 0.f : fast_exp2((float)a.gamma * __log2f(q));
    float e = dl[0];
    for (int i0 = 0; i0 < nA; i0 += kB) {
#pragma unroll
      for (int j = 0; j < kB; ++j) buf[j] = (i0 + j < nA) ? dl[(int64_t)(i0 + j) * a.d] : 0.f;
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        if (i0 + j < nA) {
          ein[(int64_t)(i0 + j) * a.d] = e;
          e = qg * e + (1.f - qg) * buf[j];
        }
      }
    }
  } else {
    // The filter's state (position, velocity, acceleration) follows the
    // linear recursion x_i = A x_{i-1} + g Delta_i, A = (I - g h) F: the
    // constant-acceleration transition F (unit step) followed by the
    // correction of the observed position (h = (1, 0, 0)) with gain g.
    const float g0 = a.corr_p[0], g1 = a.corr_p[1], g2 = a.corr_p[2];
    const float A[3][3] = {{1.f - g0, 1.f - g0, 0.5f * (1.f - g0)},
                           {-g1, 1.f - g1, 1.f - 0.5f * g1},
                           {-g2, -g2, 1.f - 0.5f * g2}};
    float x0 = dl[0], x1 = 0.f, x2 = 0.f;
    for (int i0 = 1; i0 < nA; i0 += kB) {
#pragma unroll
      for (int j = 0; j < kB; ++j) buf[j] = (i0 + j < nA) ? dl[(int64_t)(i0 + j) * a.d] : 0.f;
#pragma unroll
      for (int j = 0; j < kB; ++j) {
        if (i0 + j < nA) {
          const float y0 = A[0][0] * x0 + A[0][1] * x1 + A[0][2] * x2 + g0 * buf[j];
          const float y1 = A[1][0] * x0 + A[1][1] * x1 + A[1][2] * x2 + g1 * buf[j];
          const float y2 = A[2][0] * x0 + A[2][1] * x1 + A[2][2] * x2 + g2 * buf[j];
          x0 = y0;
          x1 = y1;
          x2 = y2;
          dl[(int64_t)(i0 + j) * a.d] = x0;
        }
      }
    }
  }
}

// Adds the per-row correction of a smoothing variant to the gamma rows of one
// group, for a range of heads (rows a_i .. a_i+gamma-1, Hq*d contiguous values
// each):  interpolation (1-beta_k) Delta_i + beta_k Delta_{i+1} with
// beta_k = k/(gamma-1) (Delta_{i+1} = Delta_i for the last group); EMA
// q^(k+1) Ein_i + (1 - q^(k+1)) Delta_i; filter: the filtered Delta_i.
template <int D, int CORR>
__global__ __launch_bounds__(kEpiThreads) void corr_apply_kernel(Args a) {
  __shared__ float c0[8192];
  __shared__ float c1[8192];
  const int tid = threadIdx.x;
  int64_t lid = blockIdx.x;
  const int n_hc = (a.Hq + a.head_chunk - 1) / a.head_chunk;
  const int hc = (int)(lid % n_hc);
  lid /= n_hc;
  const int i = (int)(lid % a.nA_max);
  const int b = (int)(lid / a.nA_max);
  const Seq sq = seq_of(a, b);
  const int nA = sq.L / a.gamma;
  if (i >= nA) return;
  const int h0 = hc * a.head_chunk;
  const int nh = min(a.Hq, h0 + a.head_chunk) - h0;
  constexpr int DC = D / 8;
  for (int idx = tid; idx < nh * DC; idx += kEpiThreads) {
    const int hh = idx / DC, dc = idx % DC;
    const int64_t row = (((int64_t)b * a.Hq + h0 + hh) * a.nA_max + i) * D + dc * 8;
    *(f32x8*)(c0 + hh * D + dc * 8) = *(const f32x8*)(a.dbuf + row);
    if (CORR == 2)
      *(f32x8*)(c1 + hh * D + dc * 8) = *(const f32x8*)(a.dbuf + row + (i + 1 < nA ? D : 0));
    if (CORR == 3) *(f32x8*)(c1 + hh * D + dc * 8) = *(const f32x8*)(a.ebuf + row);
  }
  __syncthreads();
  typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
  const int per_row = nh * DC;
  const int64_t total = (int64_t)a.gamma * per_row;
  const float lq = (CORR == 3) ? ((a.corr_p[0] >= 1.f) ? -INFINITY : __log2f(1.f - a.corr_p[0])) : 0.f;
  for (int64_t u = tid; u < total; u += kEpiThreads) {
    const int kk = (int)(u / per_row);
    const int rem = (int)(u % per_row);
    const int hh = rem / DC, dc = rem % DC;
    const f32x8 di = *(const f32x8*)(c0 + hh * D + dc * 8);
    f32x8 corr;
    if (CORR == 2) {
      const float beta = a.gamma > 1 ? (float)kk / (float)(a.gamma - 1) : 0.f;
      corr = (1.f - beta) * di + beta * *(const f32x8*)(c1 + hh * D + dc * 8);
    } else if (CORR == 3) {
      const float w = fast_exp2((float)(kk + 1) * lq);  // q^(k+1)
      corr = w * *(const f32x8*)(c1 + hh * D + dc * 8) + (1.f - w) * di;
    } else {
      corr = di;
    }
    uint16_t* p = a.out + ((sq.base + (int64_t)i * a.gamma + kk) * a.Hq + h0 + hh) * (int64_t)D + dc * 8;
    const bf16x8_t x = *(const bf16x8_t*)p;
    *(bf16x8_t*)p = __builtin_convertvector(__builtin_convertvector(x, f32x8) + corr, bf16x8_t);
  }
}

// Counts violations of what the other kernels take on trust in device-resident
// inputs (one workgroup; a debugging aid, not on the hot path):
//   cu_seqlens: starts at 0, non-decreasing, every length <= max_seqlen;
//   key-block lists, per (sequence, kv head): offsets inside [0, nnz] and
//   non-decreasing over the query blocks, each list strictly ascending.
// Every load is guarded by the checks before it, so malformed offsets are
// counted, never followed out of bounds.
__global__ __launch_bounds__(256) void check_inputs_kernel(const int32_t* cu, int B, int max_seqlen,
                                                           const int32_t* bptr,
                                                           const int32_t* bidx, int64_t nnz,
                                                           int Hkv, int nqb, int32_t* result) {
  __shared__ int32_t red[256];
  int32_t bad = 0;
  const int tid = threadIdx.x;
  if (cu) {
    if (tid == 0 && cu[0] != 0) ++bad;
    for (int i = tid; i < B; i += 256) {
      const int64_t len = (int64_t)cu[i + 1] - cu[i];
      if (len < 0 || len > max_seqlen) ++bad;
    }
  }
  if (bptr) {
    for (int64_t row = tid; row < (int64_t)B * Hkv; row += 256) {
      const int32_t* p = bptr + row * (nqb + 1);
      bool ok = p[0] >= 0 && (int64_t)p[nqb] <= nnz;
      for (int qb = 0; qb < nqb; ++qb) ok = ok && p[qb + 1] >= p[qb];
      if (!ok) {
        ++bad;
        continue;
      }
      for (int qb = 0; qb < nqb; ++qb)
        for (int64_t e = (int64_t)p[qb] + 1; e < p[qb + 1]; ++e)
          if (bidx[e] <= bidx[e - 1]) ++bad;
    }
  }
  red[tid] = bad;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) *result = red[0];
}

template <int MODE>
hipError_t launch_attn(const Args& a0, hipStream_t s, int64_t nblocks) {
  if (nblocks <= 0) return hipSuccess;
  Args a = a0;
  a.fd_rtiles = make_fastdiv((uint32_t)a.n_rtiles);
  a.fd_nC = make_fastdiv((uint32_t)(a.nC > 0 ? a.nC : 1));
  a.fd_B = make_fastdiv((uint32_t)a.B);
  a.fd_G = make_fastdiv((uint32_t)(a.Hq / a.Hkv));
  a.fd_gamma = make_fastdiv((uint32_t)a.gamma);
  a.fd_bq = make_fastdiv((uint32_t)(a.block_q > 0 ? a.block_q : 1));
  if (a.d == 128)
    hipLaunchKernelGGL((attn_kernel<128, MODE>), dim3((unsigned)nblocks), dim3(kAttnThreads), 0, s, a);
  else
    hipLaunchKernelGGL((attn_kernel<64, MODE>), dim3((unsigned)nblocks), dim3(kAttnThreads), 0, s, a);
  return hipGetLastError();
}

constexpr int kScratchDevices = 64;
std::atomic<void*> g_scratch[kScratchDevices];

}  // namespace

// Workspace of the allocation-free entry point: each device the library runs
// on holds its own copy of this array until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is a stand-in,
// not a device address): it uses the address hipGetSymbolAddress gives for
// the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

hipError_t scratch_address(int dev, void** p) {
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  void* a = g_scratch[dev].load(std::memory_order_acquire);
  if (!a) {
    const hipError_t e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!a) return hipErrorInvalidSymbol;
    g_scratch[dev].store(a, std::memory_order_release);
  }
  *p = a;
  return hipSuccess;
}

hipError_t launch_check_inputs(const int32_t* cu, int B, int max_seqlen, const int32_t* bptr,
                              const int32_t* bidx, int64_t nnz, int Hkv, int nqb,
                              int32_t* result, hipStream_t s) {
  hipLaunchKernelGGL(check_inputs_kernel, dim3(1), dim3(256), 0, s, cu, B, max_seqlen, bptr, bidx,
                     nnz, Hkv, nqb, result);
  return hipGetLastError();
}

hipError_t launch_sparse(const Args& a, hipStream_t s) {
  return launch_attn<kSparse>(a, s, (int64_t)a.B * a.n_hgroups * a.n_rtiles);
}

hipError_t launch_dense(const Args& a, hipStream_t s) {
  return launch_attn<kDense>(a, s, (int64_t)a.B * a.n_hgroups * a.n_rtiles);
}

hipError_t launch_dense_rows(const Args& a0, hipStream_t s) {
  Args a = a0;
  a.dr_n1 = a.dr_n2 = 0;
  if (!a.cu && a.nC >= 1 && a.nC <= 16 && a.gamma >= 1) {
    // Sequences of a.N tokens: the key tiles row tile rt takes from chunk c,
    // for the dense rows (anchors r * gamma, then the tail rows) as the kernel
    // decodes them.
    const int64_t nA = a.N / a.gamma, Lc = nA * a.gamma, n_rows = nA + (a.N - Lc);
    const int rpb = kRowsPerWave * a.ppw;
    const int nrt = (int)((n_rows + rpb - 1) / rpb);
    auto end = [&](int rt) {  // one past the last row's position
      const int64_t r = std::min<int64_t>((int64_t)(rt + 1) * rpb, n_rows) - 1;
      return (r < nA ? r * a.gamma : Lc + (r - nA)) + 1;
    };
    auto tiles = [&](int rt, int c) -> int64_t {
      const int64_t kc0 = (int64_t)c * a.chunk, e = end(rt);
      if (kc0 >= e) return 0;
      return (std::min<int64_t>(kc0 + a.chunk, e) + kKeyTile - 1) / kKeyTile - kc0 / kKeyTile;
    };
    a.dr_nrt = nrt;
    for (int c = 0; c < a.nC; ++c) {
      const int64_t full = nrt > 0 ? tiles(nrt - 1, c) : 0;
      int t = nrt, z = nrt;
      if (full > 0) {
        for (t = nrt; t > 0 && tiles(t - 1, c) == full;) --t;
        for (z = t; z > 0 && tiles(z - 1, c) > 0;) --z;
      }
      a.dr_t[c] = t;
      a.dr_z[c] = z;
      a.dr_n1 += nrt - t;
      a.dr_n2 += t - z;
    }
  }
  return launch_attn<kDenseRows>(a, s, (int64_t)a.B * a.n_hgroups * a.nC * a.n_rtiles);
}

hipError_t launch_delta_epilogue(const Args& a, hipStream_t s) {
  const int n_hc = (a.Hq + a.head_chunk - 1) / a.head_chunk;
  const int64_t nblocks = (int64_t)a.B * a.nR_max * n_hc;
  if (nblocks <= 0) return hipSuccess;
  const dim3 g((unsigned)nblocks), t(kEpiThreads);
#define DA_EPI(DD, E) hipLaunchKernelGGL((delta_epilogue_kernel<DD, E>), g, t, 0, s, a)
  const int epi = a.fuse ? kEpiMergeDense
                         : a.corr_mode == 0 ? kEpiDelta
                         : a.corr_mode == 1 ? kEpiRecompute : kEpiMergeOnly;
  if (a.d == 128) {
    if (epi == kEpiDelta) DA_EPI(128, kEpiDelta);
    else if (epi == kEpiRecompute) DA_EPI(128, kEpiRecompute);
    else if (epi == kEpiMergeOnly) DA_EPI(128, kEpiMergeOnly);
    else DA_EPI(128, kEpiMergeDense);
  } else {
    if (epi == kEpiDelta) DA_EPI(64, kEpiDelta);
    else if (epi == kEpiRecompute) DA_EPI(64, kEpiRecompute);
    else if (epi == kEpiMergeOnly) DA_EPI(64, kEpiMergeOnly);
    else DA_EPI(64, kEpiMergeDense);
  }
#undef DA_EPI
  return hipGetLastError();
}

// After the merge-only epilogue: the scan (EMA, filter) and the apply pass of
// the smoothing variants (modes 2-4).
hipError_t launch_correction(const Args& a, hipStream_t s) {
  if (a.corr_mode < 2) return hipSuccess;
  if (a.corr_mode >= 3) {
    const int64_t threads = (int64_t)a.B * a.Hq * a.d;
    const dim3 g((unsigned)((threads + 255) / 256)), t(256);
    if (a.corr_mode == 3)
      hipLaunchKernelGGL(corr_scan_kernel<3>, g, t, 0, s, a);
    else
      hipLaunchKernelGGL(corr_scan_kernel<4>, g, t, 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int n_hc = (a.Hq + a.head_chunk - 1) / a.head_chunk;
  const int64_t nblocks = (int64_t)a.B * a.nA_max * n_hc;
  if (nblocks <= 0) return hipSuccess;
  const dim3 g((unsigned)nblocks), t(kEpiThreads);
#define DA_APPLY(DD, C) hipLaunchKernelGGL((corr_apply_kernel<DD, C>), g, t, 0, s, a)
  if (a.d == 128) {
    if (a.corr_mode == 2) DA_APPLY(128, 2);
    else if (a.corr_mode == 3) DA_APPLY(128, 3);
    else DA_APPLY(128, 4);
  } else {
    if (a.corr_mode == 2) DA_APPLY(64, 2);
    else if (a.corr_mode == 3) DA_APPLY(64, 3);
    else DA_APPLY(64, 4);
  }
#undef DA_APPLY
  return hipGetLastError();
}

}  // namespace da
