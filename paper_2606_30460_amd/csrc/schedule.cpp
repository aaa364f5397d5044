// Per-rank instruction lists of the forward pass: the jitted code generation
// of the SAP section, with its instruction set (send / receive of q, kv, o;
// computing; the copy-and-rescale of partial outputs, here one merge per rank).
//
// Each rank computes its blocks one per stage (diagonal first, then by ring
// step, shard, chunk; a rank without a diagonal block starts at stage 1).
// Inputs come one stage ahead directly from their owner (K/V of chunk c from
// rank c, Q of shard r from rank r) into slot t % 2 of the receiver's
// double-buffered receive slots; a transferred block's partial is written to
// result slot t % 2 and returned one stage later.  Within a stage the sends
// and receives come first (all of them form one batched point-to-point
// group), then the computation, then the merge.
#include <algorithm>
#include <vector>

#include "hsap_internal.h"

using namespace hsap;

extern "C" hsap_status hsap_emit_forward(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank,
                                         hsap_op* ops, int64_t capacity, int64_t* rank_offsets,
                                         int32_t* num_stages) {
  clear_error();
  if (sp_degree < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "sp_degree %d < 1", sp_degree);
  if (!block_tiles || !exec_rank || !rank_offsets || !num_stages)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL block_tiles, exec_rank, rank_offsets or num_stages");
  if (capacity < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "capacity < 0");
  const int32_t P = sp_degree;
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c) {
      const int64_t t = block_tiles[(int64_t)r * P + c];
      const int32_t e = exec_rank[(int64_t)r * P + c];
      if (t < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "block_tiles[%d][%d] < 0", r, c);
      if (t > 0 && e != r && e != c)
        HSAP_FAIL(HSAP_ERR_INVALID_ARG, "block (%d, %d) assigned to rank %d (must be %d or %d)", r, c, e, r, c);
    }
  struct Block {
    int32_t r, c;
  };
  std::vector<std::vector<Block>> blocks((size_t)P);
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c)
      if (block_tiles[(int64_t)r * P + c] > 0) blocks[(size_t)exec_rank[(int64_t)r * P + c]].push_back(Block{r, c});
  auto ring_step = [P](const Block& b) { return ((b.r - b.c) % P + P) % P; };
  for (auto& list : blocks)
    std::sort(list.begin(), list.end(), [&](const Block& a, const Block& b) {
      const int da = a.r == a.c ? 0 : 1, db = b.r == b.c ? 0 : 1;
      if (da != db) return da < db;
      if (ring_step(a) != ring_step(b)) return ring_step(a) < ring_step(b);
      if (a.r != b.r) return a.r < b.r;
      return a.c < b.c;
    });
  // a rank without a diagonal block starts at stage 1: its first input has to arrive first
  std::vector<int32_t> first((size_t)P);
  int32_t S = 0;
  for (int32_t e = 0; e < P; ++e) {
    const auto& list = blocks[(size_t)e];
    first[(size_t)e] = !list.empty() && list[0].r == list[0].c ? 0 : 1;
    S = std::max<int32_t>(S, first[(size_t)e] + (int32_t)list.size());
  }
  // part index of chunk c in shard r: its rank among the chunks with a block of shard r
  std::vector<int32_t> part((size_t)P * P, -1), parts((size_t)P, 0);
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c)
      if (block_tiles[(int64_t)r * P + c] > 0) part[(size_t)r * P + c] = parts[(size_t)r]++;

  // ops per (rank, stage): communication and computation separately
  const size_t cells = (size_t)P * (S + 1);
  std::vector<std::vector<hsap_op>> comm(cells), comp(cells);
  auto at = [&](int32_t e, int32_t t) { return (size_t)e * (S + 1) + t; };
  for (int32_t e = 0; e < P; ++e)
    for (int32_t i = 0; i < (int32_t)blocks[(size_t)e].size(); ++i) {
      const Block b = blocks[(size_t)e][(size_t)i];
      const int32_t t = first[(size_t)e] + i;
      if (b.r == e && b.c != e) {  // K/V of chunk c from its owner, one stage ahead
        comm[at(b.c, t - 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_KV, e, t - 1, -1, b.c, -1, -1});
        comm[at(e, t - 1)].push_back(hsap_op{HSAP_OP_RECV, HSAP_T_KV, b.c, t - 1, -1, b.c, -1, t % 2});
      } else if (b.c == e && b.r != e) {  // Q of shard r from its owner; the partial returns a stage later
        comm[at(b.r, t - 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_Q, e, t - 1, b.r, -1, -1, -1});
        comm[at(e, t - 1)].push_back(hsap_op{HSAP_OP_RECV, HSAP_T_Q, b.r, t - 1, b.r, -1, -1, t % 2});
        comm[at(e, t + 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_O, b.r, t + 1, b.r, b.c, t % 2, -1});
        comm[at(b.r, t + 1)].push_back(
            hsap_op{HSAP_OP_RECV, HSAP_T_O, e, t + 1, b.r, b.c, -1, part[(size_t)b.r * P + b.c]});
      }
      const int32_t in_slot = b.r == b.c ? -1 : t % 2;
      const int32_t out_slot = b.r == e ? part[(size_t)b.r * P + b.c] : t % 2;
      comp[at(e, t)].push_back(hsap_op{HSAP_OP_COMPUTE, HSAP_T_NONE, -1, t, b.r, b.c, in_slot, out_slot});
    }
  int64_t count = 0;
  for (int32_t e = 0; e < P; ++e) {
    rank_offsets[e] = count;
    for (int32_t t = 0; t <= S; ++t) {
      auto& cm = comm[at(e, t)];
      std::sort(cm.begin(), cm.end(), [](const hsap_op& a, const hsap_op& b) {
        if (a.peer != b.peer) return a.peer < b.peer;
        if (a.op != b.op) return a.op < b.op;
        if (a.tensor != b.tensor) return a.tensor < b.tensor;
        if (a.shard != b.shard) return a.shard < b.shard;
        return a.chunk < b.chunk;
      });
      auto emit = [&](const hsap_op& o) {
        if (ops && count < capacity) ops[count] = o;
        ++count;
      };
      for (const auto& o : cm) emit(o);
      for (const auto& o : comp[at(e, t)]) emit(o);
      if (t == S && parts[(size_t)e] > 0)
        emit(hsap_op{HSAP_OP_MERGE, HSAP_T_NONE, -1, S, e, -1, -1, parts[(size_t)e]});
    }
  }
  rank_offsets[P] = count;
  *num_stages = S + 1;
  if (!ops || count > capacity)
    HSAP_FAIL(HSAP_ERR_CAPACITY, "program needs %lld ops, capacity %lld", (long long)count, (long long)capacity);
  return HSAP_OK;
}
