// da_api.cpp -- the C ABI of include/delta_attn.h: argument validation,
// workspace planning and the launch sequence of the Delta Attention prefill.
#include <math.h>
#include <string.h>

#include <cmath>

#include <atomic>

#include "delta_attn.h"
#include "da_internal.hpp"

namespace da {

namespace {

thread_local int g_last_hip_error = 0;

// Per-device answer to "is this a gfx950": 0 unknown, 1 yes, 2 no.
constexpr int kMaxDevices = 64;
std::atomic<int> g_arch_ok[kMaxDevices];
thread_local int g_cur_dev = 0;  // the device check_device() last looked at

da_status fail_hip(hipError_t e) {
  g_last_hip_error = (int)e;
  return DA_ERR_HIP;
}

da_status check_device() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e);
  if (dev < 0 || dev >= kMaxDevices) return DA_ERR_UNSUPPORTED;
  int st = g_arch_ok[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return fail_hip(e);
    st = (strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
    g_arch_ok[dev].store(st, std::memory_order_relaxed);
  }
  g_cur_dev = dev;
  return st == 1 ? DA_OK : DA_ERR_UNSUPPORTED;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

// Query heads of one GQA group that share an attention workgroup: the
// largest power of two dividing G, at most kAttnWaves.
int heads_per_block(int G) {
  int h = 1;
  while (h * 2 <= kAttnWaves && G % (h * 2) == 0) h *= 2;
  return h;
}

int fused_heads_per_block(int G, int gamma, int max_rows) {
  for (int h = heads_per_block(G); h >= 1; h /= 2) {
    const int slab = kRowsPerWave * (kAttnWaves / h);
    if (G % h == 0 && slab % gamma == 0 && slab <= max_rows) return h;
  }
  return 0;
}

// Workspace of the Delta path.  Dense rows of a sequence of length L are the
// floor(L/gamma) anchors plus the L mod gamma tail rows.  Their key axis is
// split into nC chunks of `chunk` keys (at least 2560), up to 16 of them.
// Workgroups that run at the same time then process one key chunk each in
// step with their neighbours, which keeps them sharing that chunk's keys and
// values in L2.  (The minimum sets nC only below 40960 keys.  At 32768, 13
// chunks of 2560 keys fill just under two rounds of the CUs where 16 of 2048
// filled two and a quarter: 15 % less time on the strided rows and merge.)
// nC drops only when the partial results would pass 8 GiB, or, with a nonzero
// `limit`, until the whole workspace fits `limit` bytes (false when even one
// chunk does not).
bool make_plan(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma, Plan* p, size_t limit) {
  if (B < 1 || max_seqlen < 1 || Hq < 1 || Hkv < 1 || gamma < 1 || (d != 64 && d != 128))
    return false;
  if (Hq % Hkv != 0) return false;
  const int64_t nA_max = max_seqlen / gamma;
  const int64_t nR_max = nA_max + (int64_t)((gamma - 1 < max_seqlen) ? gamma - 1 : max_seqlen);
  constexpr int64_t kMinChunkKeys = kKeyTile * 40;
  int64_t nC = (max_seqlen + kMinChunkKeys - 1) / kMinChunkKeys;
  if (nC > 16) nC = 16;
  if (nC < 1) nC = 1;
  const int64_t per_chunk_bytes = (int64_t)B * Hq * nR_max * (d + 2) * 4;
  const int64_t budget = (int64_t)8 << 30;
  while (nC > 1 && per_chunk_bytes * nC > budget) --nC;
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  auto fill = [&](int64_t want) {
    int64_t chunk = (max_seqlen + want - 1) / want;
    chunk = (chunk + kKeyTile - 1) / kKeyTile * kKeyTile;
    const int64_t n = (max_seqlen + chunk - 1) / chunk;
    p->nA_max = (int)nA_max;
    p->nR_max = (int)nR_max;
    p->nC = (int)n;
    p->chunk = (int)chunk;
    p->sa_floats = (size_t)B * Hq * nR_max * d;  // sparse anchor rows, or merged dense rows
    p->part_o_floats = (size_t)B * Hq * nR_max * n * d;
    p->part_ml_floats = (size_t)B * Hq * nR_max * n * 2;
    p->bytes = up(p->sa_floats * 4) + up(p->part_o_floats * 4) + up(p->part_ml_floats * 4);
  };
  fill(nC);
  while (limit && p->bytes > limit && p->nC > 1) fill(p->nC - 1);
  return !limit || p->bytes <= limit;
}

size_t correction_floats(int B, int max_seqlen, int Hq, int d, int gamma, int mode) {
  if (mode < 2 || gamma < 1) return 0;
  const size_t per = (size_t)B * Hq * (size_t)(max_seqlen / gamma) * d;
  return mode == 3 ? 2 * per : per;
}

namespace {

struct Problem {
  const void *q, *k, *v;
  void* out;
  const int32_t* cu;
  int B, N, Hq, Hkv, d;
  int window, n_sink, gamma;
  // key-block lists (nullptr: sink + window attention)
  const int32_t* blk_ptr = nullptr;
  const int32_t* blk_idx = nullptr;
  int block_q = 0;
};

// Rows per query head of one sparse workgroup; with key-block lists they must
// fit one query block.
int slab_rows(int hpw) { return kRowsPerWave * (kAttnWaves / hpw); }

// Shape/parameter checks shared by all calls; no HIP call happens here.
da_status validate(const Problem& P, bool need_window, bool need_gamma) {
  if (!P.q || !P.k || !P.v || !P.out) return DA_ERR_NULL;
  if (P.B < 1 || P.N < 1 || P.Hq < 1 || P.Hkv < 1 || P.Hq % P.Hkv != 0) return DA_ERR_SHAPE;
  if (need_window && (P.window < 1 || P.n_sink < 0)) return DA_ERR_PARAM;
  if (need_gamma && P.gamma < 1) return DA_ERR_PARAM;
  if (P.d != 64 && P.d != 128) return DA_ERR_UNSUPPORTED;
  // token indices and row-tile counts are 32-bit inside the kernels
  if (!P.cu && (int64_t)P.B * P.N > INT32_MAX) return DA_ERR_SHAPE;
  const int hpw = heads_per_block(P.Hq / P.Hkv);
  const int64_t rows_per_block = (int64_t)kRowsPerWave * (kAttnWaves / hpw);
  const int64_t blocks = (int64_t)P.B * (P.Hq / hpw) * ((P.N + rows_per_block - 1) / rows_per_block);
  if (blocks > INT32_MAX) return DA_ERR_SHAPE;
  if (P.blk_ptr || P.blk_idx) {
    if (!P.blk_ptr || !P.blk_idx) return DA_ERR_NULL;
    if (P.block_q != 64 && P.block_q != 128 && P.block_q != 256) return DA_ERR_PARAM;
    if (slab_rows(hpw) > P.block_q) return DA_ERR_UNSUPPORTED;
    if ((int64_t)P.B * P.Hkv * ((int64_t)(P.N + P.block_q - 1) / P.block_q + 1) > INT32_MAX)
      return DA_ERR_SHAPE;
  }
  if (!aligned16(P.q) || !aligned16(P.k) || !aligned16(P.v) || !aligned16(P.out))
    return DA_ERR_ALIGN;
  return DA_OK;
}

Args base_args(const Problem& P) {
  Args a;
  memset(&a, 0, sizeof a);
  a.q = (const uint16_t*)P.q;
  a.k = (const uint16_t*)P.k;
  a.v = (const uint16_t*)P.v;
  a.out = (uint16_t*)P.out;
  a.cu = P.cu;
  a.B = P.B;
  a.N = P.N;
  a.Hq = P.Hq;
  a.Hkv = P.Hkv;
  a.d = P.d;
  a.window = P.window;
  a.n_sink = P.n_sink;
  a.cover = (int64_t)P.n_sink + P.window;
  if (P.blk_ptr) {
    // the key set is the lists' tiles plus the own query block's, masked
    // causally: no sink/window test applies, and no anchor is known covered
    a.blk_ptr = P.blk_ptr;
    a.blk_idx = P.blk_idx;
    a.block_q = P.block_q;
    a.nqb = (P.N + P.block_q - 1) / P.block_q;
    a.n_sink = INT32_MAX;
    a.window = 1;
    a.cover = 0;
  }
  a.gamma = P.gamma > 0 ? P.gamma : 1;
  a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)P.d));
  a.hpw = heads_per_block(P.Hq / P.Hkv);
  a.ppw = kAttnWaves / a.hpw;
  a.n_hgroups = P.Hq / a.hpw;
  const int rows_per_block = kRowsPerWave * a.ppw;
  a.n_rtiles = (P.N + rows_per_block - 1) / rows_per_block;
  a.head_chunk = 8192 / P.d;
  return a;
}

da_status run_plain(const Problem& P, bool sparse, void* stream) {
  da_status st = validate(P, sparse, false);
  if (st != DA_OK) return st;
  st = check_device();
  if (st != DA_OK) return st;
  Args a = base_args(P);
  hipError_t e = sparse ? launch_sparse(a, (hipStream_t)stream) : launch_dense(a, (hipStream_t)stream);
  if (e != hipSuccess) return fail_hip(e);
  return DA_OK;
}

// Launch sequence of the Delta path.  Unfused schedule: sparse kernel (plus
// the fp32 sparse rows at anchors), strided dense rows, then the epilogue
// that merges them, forms Delta and adds it to `out` in place.  Fused
// schedule (when every group of gamma rows fits one head slab of a sparse
// workgroup, and for the Delta and recompute corrections only): strided
// dense rows, the merge into fp32 dense rows, then the sparse kernel storing
// the corrected rows.  `steps` without DA_STEP_FUSED picks the unfused
// schedule; `auto_fuse` lets the whole-path calls take the fused one.
da_status run_delta(const Problem& P, void* workspace, size_t workspace_bytes, void* stream,
                    unsigned steps, bool auto_fuse, int corr_mode = 0, float p0 = 0.f,
                    float p1 = 0.f, float p2 = 0.f, bool scratch = false) {
  da_status st = validate(P, true, true);
  if (st != DA_OK) return st;
  if ((steps & DA_STEP_ALL) == 0u || steps > (DA_STEP_ALL | DA_STEP_FUSED)) return DA_ERR_PARAM;
  if (corr_mode < DA_CORR_DELTA || corr_mode > DA_CORR_ABG) return DA_ERR_PARAM;
  if (!std::isfinite(p0) || !std::isfinite(p1) || !std::isfinite(p2)) return DA_ERR_PARAM;
  if (corr_mode == DA_CORR_EMA && (p0 < 0.f || p0 > 1.f)) return DA_ERR_PARAM;
  const int fhpw = fused_heads_per_block(P.Hq / P.Hkv, P.gamma, P.blk_ptr ? P.block_q : INT32_MAX);
  const bool can_fuse = fhpw > 0 && corr_mode <= DA_CORR_RECOMPUTE;
  if ((steps & DA_STEP_FUSED) && !can_fuse) return DA_ERR_UNSUPPORTED;
  const bool fused = (steps & DA_STEP_FUSED) || (auto_fuse && can_fuse);
  Plan plan;
  if (!make_plan(P.B, P.N, P.Hq, P.Hkv, P.d, P.gamma, &plan)) return DA_ERR_SHAPE;
  if (scratch) {
    // the static scratch array: as many key chunks as fit it
    if (!make_plan(P.B, P.N, P.Hq, P.Hkv, P.d, P.gamma, &plan, kScratchBytes))
      return DA_ERR_WORKSPACE;
  } else {
    const size_t extra = correction_floats(P.B, P.N, P.Hq, P.d, P.gamma, corr_mode) * 4;
    if (!workspace || workspace_bytes < plan.bytes + extra) return DA_ERR_WORKSPACE;
    if (!aligned16(workspace)) return DA_ERR_ALIGN;
  }
  {
    const int hpw = heads_per_block(P.Hq / P.Hkv);
    const int64_t rows_per_block = (int64_t)kRowsPerWave * (kAttnWaves / hpw);
    const int64_t rtiles = (plan.nR_max + rows_per_block - 1) / rows_per_block;
    if ((int64_t)P.B * (P.Hq / hpw) * plan.nC * rtiles > INT32_MAX) return DA_ERR_SHAPE;
    if ((int64_t)P.B * plan.nR_max * ((P.Hq + 8192 / P.d - 1) / (8192 / P.d)) > INT32_MAX)
      return DA_ERR_SHAPE;
    if (fused) {
      const int64_t frows = (int64_t)kRowsPerWave * (kAttnWaves / fhpw);
      if ((int64_t)P.B * (P.Hq / fhpw) * ((P.N + frows - 1) / frows) > INT32_MAX)
        return DA_ERR_SHAPE;
    }
  }
  st = check_device();
  if (st != DA_OK) return st;
  if (scratch) {
    // this device's copy of the static array (its address is looked up once
    // per device, with the device current)
    const hipError_t e = scratch_address(g_cur_dev, &workspace);
    if (e != hipSuccess) return fail_hip(e);
  }

  Args a = base_args(P);
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  char* ws = (char*)workspace;
  a.sa = (float*)ws;
  a.part_o = (float*)(ws + up(plan.sa_floats * 4));
  a.part_ml = (float*)(ws + up(plan.sa_floats * 4) + up(plan.part_o_floats * 4));
  a.nA_max = plan.nA_max;
  a.nR_max = plan.nR_max;
  a.nC = plan.nC;
  a.chunk = plan.chunk;
  a.corr_mode = corr_mode;
  a.corr_p[0] = p0;
  a.corr_p[1] = p1;
  a.corr_p[2] = p2;
  if (corr_mode >= DA_CORR_INTERP) {
    a.dbuf = (float*)(ws + plan.bytes);
    a.ebuf = a.dbuf + (size_t)P.B * P.Hq * (size_t)plan.nA_max * P.d;
  }
  hipStream_t s = (hipStream_t)stream;

  hipError_t e = hipSuccess;
  if (fused) {
    a.dense = a.sa;
    a.fuse = corr_mode == DA_CORR_RECOMPUTE ? 2 : 1;
    if (steps & DA_STEP_DENSE_ROWS) {
      Args ar = a;
      ar.n_rtiles = (plan.nR_max + kRowsPerWave * a.ppw - 1) / (kRowsPerWave * a.ppw);
      e = launch_dense_rows(ar, s);
      if (e != hipSuccess) return fail_hip(e);
    }
    if (steps & DA_STEP_CORRECT) {
      e = launch_delta_epilogue(a, s);
      if (e != hipSuccess) return fail_hip(e);
    }
    if (steps & DA_STEP_SPARSE) {
      Args as = a;
      as.hpw = fhpw;
      as.ppw = kAttnWaves / fhpw;
      as.n_hgroups = P.Hq / fhpw;
      as.n_rtiles = (P.N + kRowsPerWave * as.ppw - 1) / (kRowsPerWave * as.ppw);
      e = launch_sparse(as, s);
      if (e != hipSuccess) return fail_hip(e);
    }
    return DA_OK;
  }
  // Step 1: sparse attention for every row (+ fp32 copy at anchors).
  if (steps & DA_STEP_SPARSE) {
    e = launch_sparse(a, s);
    if (e != hipSuccess) return fail_hip(e);
  }
  // Steps 2-3: dense attention at anchors and tail rows, key axis split in chunks.
  if (steps & DA_STEP_DENSE_ROWS) {
    Args ar = a;
    ar.n_rtiles = (plan.nR_max + kRowsPerWave * a.ppw - 1) / (kRowsPerWave * a.ppw);
    e = launch_dense_rows(ar, s);
    if (e != hipSuccess) return fail_hip(e);
  }
  // Steps 4-5: merge, Delta, broadcast-add in place (or the chosen variant).
  if (steps & DA_STEP_CORRECT) {
    e = launch_delta_epilogue(a, s);
    if (e != hipSuccess) return fail_hip(e);
    e = launch_correction(a, s);
    if (e != hipSuccess) return fail_hip(e);
  }
  return DA_OK;
}

}  // namespace
}  // namespace da

using da::Problem;

extern "C" {

da_status delta_attn_prefill(const void* q, const void* k, const void* v, void* out, int B,
                             int Hq, int Hkv, int N, int d, int window, int n_sink, int gamma,
                             void* workspace, size_t workspace_bytes, void* stream) {
  Problem P{q, k, v, out, nullptr, B, N, Hq, Hkv, d, window, n_sink, gamma};
  return da::run_delta(P, workspace, workspace_bytes, stream, DA_STEP_ALL, true);
}

da_status delta_attn_prefill_varlen(const void* q, const void* k, const void* v, void* out,
                                    const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                    int Hkv, int d, int window, int n_sink, int gamma,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  if (!cu_seqlens) return DA_ERR_NULL;
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, window, n_sink, gamma};
  return da::run_delta(P, workspace, workspace_bytes, stream, DA_STEP_ALL, true);
}

da_status delta_attn_prefill_steps(const void* q, const void* k, const void* v, void* out,
                                   const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                   int Hkv, int d, int window, int n_sink, int gamma,
                                   void* workspace, size_t workspace_bytes, void* stream,
                                   unsigned steps) {
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, window, n_sink, gamma};
  return da::run_delta(P, workspace, workspace_bytes, stream, steps, false);
}

da_status delta_attn_prefill_correction(const void* q, const void* k, const void* v, void* out,
                                        const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                        int Hkv, int d, int window, int n_sink, int gamma,
                                        int mode, float p0, float p1, float p2, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, window, n_sink, gamma};
  return da::run_delta(P, workspace, workspace_bytes, stream, DA_STEP_ALL, true, mode, p0, p1,
                       p2);
}

da_status delta_attn_prefill_noalloc(const void* q, const void* k, const void* v, void* out,
                                     const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                     int Hkv, int d, int window, int n_sink, int gamma,
                                     void* stream) {
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, window, n_sink, gamma};
  return da::run_delta(P, nullptr, 0, stream, DA_STEP_ALL, true, 0, 0.f, 0.f, 0.f, true);
}

size_t da_workspace_bytes_correction(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma,
                                     int mode) {
  da::Plan p;
  if (mode < DA_CORR_DELTA || mode > DA_CORR_ABG) return 0;
  if (!da::make_plan(B, max_seqlen, Hq, Hkv, d, gamma, &p)) return 0;
  return p.bytes + da::correction_floats(B, max_seqlen, Hq, d, gamma, mode) * 4;
}

da_status sparse_attn_prefill(const void* q, const void* k, const void* v, void* out, int B,
                              int Hq, int Hkv, int N, int d, int window, int n_sink,
                              void* stream) {
  Problem P{q, k, v, out, nullptr, B, N, Hq, Hkv, d, window, n_sink, 1};
  return da::run_plain(P, true, stream);
}

da_status sparse_attn_prefill_varlen(const void* q, const void* k, const void* v, void* out,
                                     const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                     int Hkv, int d, int window, int n_sink, void* stream) {
  if (!cu_seqlens) return DA_ERR_NULL;
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, window, n_sink, 1};
  return da::run_plain(P, true, stream);
}

da_status dense_causal_attn_prefill(const void* q, const void* k, const void* v, void* out,
                                    int B, int Hq, int Hkv, int N, int d, void* stream) {
  Problem P{q, k, v, out, nullptr, B, N, Hq, Hkv, d, 1, 0, 1};
  return da::run_plain(P, false, stream);
}

da_status dense_causal_attn_prefill_varlen(const void* q, const void* k, const void* v,
                                           void* out, const int32_t* cu_seqlens, int B,
                                           int max_seqlen, int Hq, int Hkv, int d,
                                           void* stream) {
  if (!cu_seqlens) return DA_ERR_NULL;
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, 1, 0, 1};
  return da::run_plain(P, false, stream);
}

int da_fused_supported(int Hq, int Hkv, int gamma) {
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || gamma < 1) return 0;
  return da::fused_heads_per_block(Hq / Hkv, gamma, INT32_MAX) > 0 ? 1 : 0;
}

int da_fused_supported_blocksparse(int Hq, int Hkv, int gamma, int block_q) {
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || gamma < 1) return 0;
  if (block_q != 64 && block_q != 128 && block_q != 256) return 0;
  return da::fused_heads_per_block(Hq / Hkv, gamma, block_q) > 0 ? 1 : 0;
}

da_status blocksparse_attn_prefill(const void* q, const void* k, const void* v, void* out,
                                   const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                   int Hkv, int d, int block_q, const int32_t* block_ptr,
                                   const int32_t* block_idx, void* stream) {
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, 1, 0, 1};
  P.blk_ptr = block_ptr;
  P.blk_idx = block_idx;
  P.block_q = block_q;
  if (!block_ptr || !block_idx) return DA_ERR_NULL;
  return da::run_plain(P, true, stream);
}

da_status delta_attn_prefill_blocksparse(const void* q, const void* k, const void* v, void* out,
                                         const int32_t* cu_seqlens, int B, int max_seqlen,
                                         int Hq, int Hkv, int d, int block_q,
                                         const int32_t* block_ptr, const int32_t* block_idx,
                                         int gamma, void* workspace, size_t workspace_bytes,
                                         void* stream, unsigned steps) {
  Problem P{q, k, v, out, cu_seqlens, B, max_seqlen, Hq, Hkv, d, 1, 0, gamma};
  P.blk_ptr = block_ptr;
  P.blk_idx = block_idx;
  P.block_q = block_q;
  if (!block_ptr || !block_idx) return DA_ERR_NULL;
  if (steps == 0u) return da::run_delta(P, workspace, workspace_bytes, stream, DA_STEP_ALL, true);
  return da::run_delta(P, workspace, workspace_bytes, stream, steps, false);
}

da_status da_launch_plan(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma, int block_q,
                         da_plan* plan) {
  if (!plan) return DA_ERR_NULL;
  if (B < 1 || max_seqlen < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return DA_ERR_SHAPE;
  if (gamma < 1) return DA_ERR_PARAM;
  if (block_q != 0 && block_q != 64 && block_q != 128 && block_q != 256) return DA_ERR_PARAM;
  if (d != 64 && d != 128) return DA_ERR_UNSUPPORTED;
  da::Plan p;
  if (!da::make_plan(B, max_seqlen, Hq, Hkv, d, gamma, &p)) return DA_ERR_SHAPE;
  const int G = Hq / Hkv;
  const int hpw = da::heads_per_block(G);
  if (block_q && da::kRowsPerWave * (da::kAttnWaves / hpw) > block_q) return DA_ERR_UNSUPPORTED;
  const int fhpw = da::fused_heads_per_block(G, gamma, block_q ? block_q : INT32_MAX);
  plan->fused = fhpw > 0 ? 1 : 0;
  plan->sparse_heads = fhpw > 0 ? fhpw : hpw;
  plan->sparse_slab_rows = da::kRowsPerWave * (da::kAttnWaves / (fhpw > 0 ? fhpw : hpw));
  plan->rows_heads = hpw;
  plan->key_chunks = p.nC;
  plan->chunk_keys = p.chunk;
  plan->key_tile = da::kKeyTile;
  plan->rows_per_wave = da::kRowsPerWave;
  plan->waves_per_block = da::kAttnWaves;
  return DA_OK;
}

size_t da_workspace_bytes(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma) {
  da::Plan p;
  if (!da::make_plan(B, max_seqlen, Hq, Hkv, d, gamma, &p)) return 0;
  return p.bytes;
}

da_status da_check_inputs(const int32_t* cu_seqlens, int B, int max_seqlen, int Hkv,
                          int block_q, const int32_t* block_ptr, const int32_t* block_idx,
                          int64_t block_nnz, int32_t* result, void* stream) {
  if (!result || (!cu_seqlens && !block_ptr)) return DA_ERR_NULL;
  if (B < 1 || max_seqlen < 1) return DA_ERR_SHAPE;
  int nqb = 0;
  if (block_ptr) {
    if (!block_idx && block_nnz > 0) return DA_ERR_NULL;
    if (Hkv < 1 || block_nnz < 0) return DA_ERR_SHAPE;
    if (block_q != 64 && block_q != 128 && block_q != 256) return DA_ERR_PARAM;
    nqb = (max_seqlen + block_q - 1) / block_q;
  }
  if (((uintptr_t)result & 3u) != 0) return DA_ERR_ALIGN;
  da_status st = da::check_device();
  if (st != DA_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = da::launch_check_inputs(cu_seqlens, B, max_seqlen, block_ptr, block_idx,
                                         block_nnz, Hkv, nqb, result, s);
  if (e != hipSuccess) return da::fail_hip(e);
  int32_t host = 0;
  e = hipMemcpyAsync(&host, result, sizeof host, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return da::fail_hip(e);
  return host == 0 ? DA_OK : DA_ERR_PARAM;
}

const char* da_status_string(da_status s) {
  switch (s) {
    case DA_OK: return "DA_OK";
    case DA_ERR_NULL: return "DA_ERR_NULL";
    case DA_ERR_SHAPE: return "DA_ERR_SHAPE";
    case DA_ERR_PARAM: return "DA_ERR_PARAM";
    case DA_ERR_UNSUPPORTED: return "DA_ERR_UNSUPPORTED";
    case DA_ERR_ALIGN: return "DA_ERR_ALIGN";
    case DA_ERR_WORKSPACE: return "DA_ERR_WORKSPACE";
    case DA_ERR_HIP: return "DA_ERR_HIP";
  }
  return "DA_ERR_UNKNOWN";
}

int da_last_hip_error(void) { return da::g_last_hip_error; }

int da_abi_version(void) { return DA_ABI_VERSION; }

}  // extern "C"
