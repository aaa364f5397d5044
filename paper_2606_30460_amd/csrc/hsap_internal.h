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
// A batch of B packed sequences of Ns tokens each, concatenated (sequence b
// holds positions b*Ns .. b*Ns+Ns-1), every sequence split P ways.  Shard
// (or chunk) x holds ns = Ns/P positions of each sequence; its local rows are
// b*ns + l.  CONTIGUOUS: position b*Ns + x*ns + l.  ZIGZAG: each sequence is
// cut into 2P pieces of m = Ns/(2P); rows l < m are piece x, rows m..2m-1 are
// piece 2P-1-x.
// ---------------------------------------------------------------------------
struct Geom {
  int64_t N;   // positions over the batch (B * Ns)
  int64_t n;   // rows per shard over the batch (B * ns)
  int64_t m;   // rows per piece of one sequence (ns for CONTIGUOUS, ns/2 for ZIGZAG)
  int64_t Ns;  // tokens per sequence
  int64_t ns;  // rows per shard of one sequence
  int32_t P;
  int32_t layout;
  int32_t B;
};

HSAP_HD inline int64_t global_pos(const Geom& g, int32_t shard, int64_t local) {
  int64_t base = 0;
  if (g.B > 1) {  // rows and positions stay below 2^31 (checked with the descriptor)
    const uint32_t b = (uint32_t)local / (uint32_t)g.ns;
    base = (int64_t)b * g.Ns;
    local -= (int64_t)b * g.ns;
  }
  if (g.layout == HSAP_LAYOUT_CONTIGUOUS) return base + (int64_t)shard * g.ns + local;
  return base + (local < g.m ? (int64_t)shard * g.m + local : (int64_t)(2 * g.P - 1 - shard) * g.m + (local - g.m));
}

// Validates N, P, layout, shard id and tile sizes; fills `g`.
hsap_status check_shard(const hsap_shard_desc* d, Geom* g);

// Validates an attention descriptor (shard part plus heads, head_dim, scale).
hsap_status check_attn(const hsap_attn_desc* d, Geom* g);

// Whether the backward kernels exist for the descriptor's (head_dim, BM, BN); the descriptor
// must already pass check_attn.
bool backward_supported(const hsap_attn_desc* d);

#if defined(__HIPCC__)
// First index i of tiles[0 .. num - 1] (sorted by q_tile) with tiles[i].q_tile >= key, for the
// tile-list entry points (one chunk's tiles in the planner's order).  Wave-wide: each round
// narrows the range 64-fold with one strided probe per lane, the last compares a window of at
// most 64 entries; every probe stays inside the list (num <= 2^30).  The result is the same on
// every lane.
__device__ inline int32_t lower_bound_q_tile(const hsap_tile* tiles, int32_t num, int32_t key, int lane) {
  if (num <= 0) return 0;
  int32_t lo = 0, len = num;
  while (len > 64) {
    const int32_t stride = (len + 63) >> 6;
    const int32_t idx = min(lo + lane * stride, lo + len - 1);
    const bool below = lo + lane * stride < lo + len && tiles[idx].q_tile < key;
    const int32_t cnt = __popcll(__builtin_amdgcn_ballot_w64(below));
    if (cnt == 0) return lo;  // tiles[lo] is already >= key
    const int32_t next = lo + (cnt - 1) * stride + 1;
    len = min(lo + cnt * stride, lo + len) - next;
    lo = next;
  }
  const bool below = lane < len && tiles[min(lo + lane, num - 1)].q_tile < key;
  return lo + __popcll(__builtin_amdgcn_ballot_w64(below));
}

// Workgroup bid of a (run, query head) grid -> its run and query head.  Workgroups are dispatched
// to the eight XCDs round-robin (workgroup i on XCD i % 8), and each XCD has its own L2.  When the
// K/V heads split evenly over the XCDs, the query heads that read one K/V head are placed on one
// XCD (K/V head g on XCD g % 8), so the K/V tiles they share are fetched into one L2 instead of
// `group` of them.  Runs keep their order (longest first) on every XCD.  Without grouped heads
// (hq == hkv) this is the plain run-major order, head fastest.
__device__ inline void run_and_head(int bid, int hq, int hkv, int& run, int& h) {
  if (hkv % 8 == 0 && hq != hkv) {
    const int per = hq >> 3;  // query heads per XCD
    const int group = hq / hkv;
    const int x = bid & 7, y = bid >> 3;
    run = y / per;
    const int lh = y - run * per;  // the XCD's lh-th query head: K/V head 8 j + x, member i
    const int j = lh / group, i = lh - j * group;
    h = (8 * j + x) * group + i;
  } else {
    run = bid / hq;
    h = bid - run * hq;
  }
}

// The run of q-tile qt in a sorted tile list: {slot 0, qt, first, count}.
__device__ inline hsap_run q_tile_run(const hsap_tile* tiles, int32_t num, int32_t qt, int lane) {
  const int32_t first = lower_bound_q_tile(tiles, num, qt, lane);
  const int32_t end = lower_bound_q_tile(tiles, num, qt + 1, lane);
  return hsap_run{0, qt, first, end - first};
}

// Workgroups of the bf16 partial forward resident on one compute unit for the descriptor's shape
// (the runtime's occupancy of the kernel that runs); 0 when there is none.
int fwd_resident_per_cu(const hsap_attn_desc* d);
#endif

#if defined(__HIPCC__)
// Zeroes tiles tiles[0 .. num_tiles-1] (device int32) of both a and b, tile t being the byte
// range [t * tile_bytes, (t + 1) * tile_bytes); tile_bytes a multiple of 16, a and b 16-byte
// aligned.  Nothing is launched for an empty list.
hsap_status zero_tiles(void* a, void* b, const int32_t* tiles, int32_t num_tiles, int64_t tile_bytes,
                       hipStream_t stream);

// hsap_lse_merge over the rows of the BM-row q-tiles listed in tiles[0 .. num_tiles-1] (device
// int32), or over every row when tiles is NULL; rows of other q-tiles are neither read nor written.
hsap_status lse_merge(int32_t num_parts, const float* const* o_parts, const float* const* lse_parts, int64_t n,
                      int32_t heads_q, int32_t head_dim, void* o_out, float* lse_out, const int32_t* tiles,
                      int32_t num_tiles, int32_t block_m, hipStream_t stream);

// The executor's forwards.  Document starts come from the cumulative lengths cu_seqlens
// [num_docs + 1] on the device (no per-position start array).  fused: hsap_attn_fwd_fused over
// runs that span every chunk.  Otherwise hsap_partial_attn_fwd_runs, where runs whose slot is
// kFinalSlot write the final bf16 O and LSE of their q-tile to o_out / lse_out (the q-tile's
// only part: nothing to merge).
constexpr int32_t kFinalSlot = -2;

// hsap_attn_bwd_bf16 with the backward preprocess folded into the dQ kernel: delta (device fp32
// [Hq, n], written) is computed there from o and d_o, and read by the dK/dV kernel launched after.
hsap_status attn_bwd_bf16_delta(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                const void* d_o, const void* o, const float* lse, float* delta,
                                const int32_t* doc_start, const hsap_tile* tiles_k, const hsap_run* runs_k,
                                int64_t num_runs_k, const hsap_tile* tiles_q, const hsap_run* runs_q,
                                int64_t num_runs_q, void* dq, void* dk, void* dv, hipStream_t stream);
hsap_status executor_forward(const hsap_attn_desc* desc, bool fused, const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens, int32_t num_docs, const hsap_tile* tiles,
                             const hsap_run* runs, int64_t num_runs, float* o_part, float* lse_part,
                             int32_t num_slots, void* o_out, float* lse_out, hipStream_t stream);
#endif

}  // namespace hsap
