// Internal declarations shared by the libhsap translation units (not installed).
#pragma once

#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/hsap.h"

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
#define HSAP_HD __host__ __device__
#else
#define HSAP_HD
#endif

namespace hsap {

// ---------------------------------------------------------------------------
// error reporting (thread-local message behind hsap_last_error)
// ---------------------------------------------------------------------------
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

#define HSAP_FAIL(code, ...)        \
  do {                              \
    ::hsap::set_error(__VA_ARGS__); \
    return code;                    \
  } while (0)

// ---------------------------------------------------------------------------
// shard geometry
//
// Shard (or chunk) x of a sequence of N tokens split P ways holds n = N/P
// positions.  CONTIGUOUS: x*n + l.  ZIGZAG: the sequence is cut into 2P
// pieces of m = N/(2P); local rows 0..m-1 are piece x, rows m..2m-1 are
// piece 2P-1-x.
// ---------------------------------------------------------------------------
struct Geom {
  int64_t N;
  int64_t n;  // rows per shard
  int64_t m;  // rows per piece (n for CONTIGUOUS, n/2 for ZIGZAG)
  int32_t P;
  int32_t layout;
};

HSAP_HD inline int64_t global_pos(const Geom& g, int32_t shard, int64_t local) {
  if (g.layout == HSAP_LAYOUT_CONTIGUOUS) return (int64_t)shard * g.n + local;
  return local < g.m ? (int64_t)shard * g.m + local : (int64_t)(2 * g.P - 1 - shard) * g.m + (local - g.m);
}

// Validates N, P, layout, shard id and tile sizes; fills `g`.
hsap_status check_shard(const hsap_shard_desc* d, Geom* g);

// Validates an attention descriptor (shard part plus heads, head_dim, scale).
hsap_status check_attn(const hsap_attn_desc* d, Geom* g);

#if defined(__HIPCC__)
// Writes `bytes` zero bytes at dst on `stream` with a kernel (bytes a multiple
// of 4, dst 16-byte aligned).
hsap_status zero_fill(void* dst, int64_t bytes, hipStream_t stream);
#endif

}  // namespace hsap
