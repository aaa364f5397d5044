// Sum of gradient parts: the accumulation step of the backward's per-rank
// programs.  A rank receives the dQ parts of its shard (one per chunk its
// queries meet) and the dK/dV parts of its chunk (one per shard whose queries
// meet it) from the ranks that computed them, and adds them up in part order.
// HBM-bound: every part is read once, the sum written once.
#include <algorithm>

#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

struct SumArgs {
  const float* part[HSAP_MAX_MERGE_PARTS];
  int32_t num_parts;
  int64_t count;
  float* out32;
  __bf16* out16;
};

// Four consecutive elements per thread per iteration (16-byte loads), grid-stride.  The parts are
// added left to right, starting from part 0, in fp32.
__global__ __launch_bounds__(256) void sum_parts_kernel(SumArgs a) {
  const int64_t quads = a.count / 4;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < quads; i += stride) {
    f32x4 acc = *(const f32x4*)(a.part[0] + 4 * i);
    for (int p = 1; p < a.num_parts; ++p) acc = acc + *(const f32x4*)(a.part[p] + 4 * i);
    if (a.out16) {
      *(bf16x4*)(a.out16 + 4 * i) = bf16x4{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
    } else {
      *(f32x4*)(a.out32 + 4 * i) = acc;
    }
  }
  // the last count % 4 elements, one per thread of the first block
  const int64_t tail = quads * 4 + threadIdx.x;
  if (blockIdx.x == 0 && threadIdx.x < 4 && tail < a.count) {
    float acc = a.part[0][tail];
    for (int p = 1; p < a.num_parts; ++p) acc = acc + a.part[p][tail];
    if (a.out16) a.out16[tail] = (__bf16)acc;
    else a.out32[tail] = acc;
  }
}

}  // namespace hsap

using namespace hsap;

extern "C" hsap_status hsap_sum_parts(int32_t num_parts, const float* const* parts, int64_t count, void* out,
                                      int32_t out_bf16, void* hip_stream) {
  clear_error();
  if (num_parts < 1 || num_parts > HSAP_MAX_MERGE_PARTS)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_parts %d outside 1..%d", num_parts, HSAP_MAX_MERGE_PARTS);
  if (count < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "count %lld < 0", (long long)count);
  if (!parts || !out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  SumArgs a{};
  for (int p = 0; p < num_parts; ++p) {
    if (!parts[p]) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "part %d is NULL", p);
    if ((uintptr_t)parts[p] & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "part %d not 16-byte aligned", p);
    a.part[p] = parts[p];
  }
  if ((uintptr_t)out & (out_bf16 ? 7 : 15)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "out not %d-byte aligned", out_bf16 ? 8 : 16);
  if (count == 0) return HSAP_OK;
  a.num_parts = num_parts;
  a.count = count;
  if (out_bf16) a.out16 = (__bf16*)out;
  else a.out32 = (float*)out;
  const int64_t blocks = std::min<int64_t>(std::max<int64_t>((count / 4 + 255) / 256, 1), 8192);
  hipLaunchKernelGGL(sum_parts_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)hip_stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "sum_parts launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}
