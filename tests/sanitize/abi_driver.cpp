// Calls the C ABI's entry points with arguments validation must reject, on
// host memory that stands in for the tensors, and checks the status codes and
// that nothing was written.  Built together with the library's host layer
// (da_api.cpp, compiled for the host only) under AddressSanitizer and
// UndefinedBehaviorSanitizer by tests/test_sanitizers.py; the kernel launchers
// are stubs that must never be reached.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "delta_attn.h"
#include "da_internal.hpp"

namespace da {
static int g_launched = 0;
hipError_t launch_sparse(const Args&, hipStream_t) { ++g_launched; return hipSuccess; }
hipError_t launch_dense(const Args&, hipStream_t) { ++g_launched; return hipSuccess; }
hipError_t launch_dense_rows(const Args&, hipStream_t) { ++g_launched; return hipSuccess; }
hipError_t launch_delta_epilogue(const Args&, hipStream_t) { ++g_launched; return hipSuccess; }
hipError_t launch_correction(const Args&, hipStream_t) { ++g_launched; return hipSuccess; }
hipError_t scratch_address(int, void** p) {
  ++g_launched;
  *p = nullptr;
  return hipSuccess;
}
hipError_t launch_check_inputs(const int32_t*, int, int, const int32_t*, const int32_t*, int64_t,
                               int, int, int32_t*, hipStream_t) {
  ++g_launched;
  return hipSuccess;
}
}  // namespace da

static int failures = 0;
static void expect(int got, int want, const char* what) {
  if (got != want) {
    fprintf(stderr, "%s: status %d, expected %d\n", what, got, want);
    ++failures;
  }
}

int main() {
  std::vector<unsigned char> buf(1 << 16, 0x5A);
  unsigned char* p = buf.data() + ((16 - (uintptr_t)buf.data() % 16) % 16);
  const std::vector<unsigned char> before = buf;
  int32_t lists[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  expect(delta_attn_prefill(nullptr, p, p, p, 1, 8, 2, 64, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_NULL, "null q");
  expect(delta_attn_prefill(p, p, p, p, 0, 8, 2, 64, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_SHAPE, "B 0");
  expect(delta_attn_prefill(p, p, p, p, 1, 6, 4, 64, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_SHAPE, "Hq % Hkv");
  expect(delta_attn_prefill(p, p, p, p, 70000, 8, 2, 70000, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_SHAPE, "T overflow");
  expect(delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 0, 4, 16, p, 1 << 20, nullptr), DA_ERR_PARAM, "window 0");
  expect(delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 16, -1, 16, p, 1 << 20, nullptr), DA_ERR_PARAM, "sinks < 0");
  expect(delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 80, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_UNSUPPORTED, "d 80");
  expect(delta_attn_prefill(p + 2, p, p, p, 1, 8, 2, 64, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_ALIGN, "align q");
  expect(delta_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 16, 4, 16, p, 100, nullptr), DA_ERR_WORKSPACE, "workspace");
  expect(delta_attn_prefill_varlen(p, p, p, p, nullptr, 2, 64, 8, 2, 128, 16, 4, 16, p, 1 << 20, nullptr), DA_ERR_NULL, "varlen cu");
  expect(delta_attn_prefill_steps(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 16, 4, 16, p, 1 << 20, nullptr, 0), DA_ERR_PARAM, "steps 0");
  expect(delta_attn_prefill_steps(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 16, 4, 16, p, 1 << 20, nullptr, 32), DA_ERR_PARAM, "steps 32");
  expect(delta_attn_prefill_correction(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 16, 4, 16, 7, 0.f, 0.f, 0.f, p, 1 << 20, nullptr), DA_ERR_PARAM, "mode 7");
  expect(delta_attn_prefill_correction(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 16, 4, 16, 3, 2.f, 0.f, 0.f, p, 1 << 20, nullptr), DA_ERR_PARAM, "ema 2");
  expect(blocksparse_attn_prefill(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 96, lists, lists, nullptr), DA_ERR_PARAM, "block_q 96");
  expect(blocksparse_attn_prefill(p, p, p, p, nullptr, 1, 64, 2, 2, 128, 64, lists, lists, nullptr), DA_ERR_UNSUPPORTED, "slab > block_q");
  expect(delta_attn_prefill_blocksparse(p, p, p, p, nullptr, 1, 64, 8, 2, 128, 64, nullptr, lists, 16, p, 1 << 20, nullptr, 0), DA_ERR_NULL, "no lists");
  expect(sparse_attn_prefill(p, p, p, p, 1, 8, 2, 64, 128, 16, -2, nullptr), DA_ERR_PARAM, "sparse sinks");
  expect(dense_causal_attn_prefill(p, p, p, p, 1, 8, 2, 64, 256, nullptr), DA_ERR_UNSUPPORTED, "dense d 256");
  int32_t* rp = (int32_t*)p;
  expect(da_check_inputs(nullptr, 2, 64, 2, 64, nullptr, nullptr, 0, rp, nullptr), DA_ERR_NULL, "check: nothing");
  expect(da_check_inputs(lists, 2, 64, 2, 64, nullptr, nullptr, 0, nullptr, nullptr), DA_ERR_NULL, "check: result");
  expect(da_check_inputs(lists, 0, 64, 2, 64, nullptr, nullptr, 0, rp, nullptr), DA_ERR_SHAPE, "check: B");
  expect(da_check_inputs(nullptr, 1, 64, 2, 100, lists, lists, 8, rp, nullptr), DA_ERR_PARAM, "check: block_q");
  expect(da_workspace_bytes(1, 64, 8, 3, 128, 16) == 0 ? 0 : 1, 0, "workspace of a bad shape");
  expect(da_workspace_bytes(1, 1 << 20, 32, 8, 128, 64) % 256 == 0 ? 0 : 1, 0, "workspace alignment");
  expect(da_fused_supported(32, 8, 64), 1, "fused 64");
  expect(da_fused_supported_blocksparse(8, 8, 16, 128), 0, "fused blocksparse");
  expect(strcmp(da_status_string(DA_ERR_HIP), "DA_ERR_HIP") == 0 ? 0 : 1, 0, "status string");
  if (buf != before) { fprintf(stderr, "a rejected call wrote to its buffers\n"); ++failures; }
  if (da::g_launched) { fprintf(stderr, "a rejected call reached a kernel launcher\n"); ++failures; }
  if (failures) return 1;
  printf("abi driver ok\n");
  return 0;
}
