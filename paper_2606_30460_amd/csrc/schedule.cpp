// Per-rank instruction lists of the forward and the backward pass: the jitted
// code generation of the SAP section, with its instruction set (send / receive
// of q, kv, o, dq, dkv, do; computing; local copies -- here the
// copy-and-rescale of partial outputs as one merge per rank, and the
// accumulation of gradient parts as one sum per rank).
//
// Each rank computes its blocks one per stage (diagonal first, then by ring
// step, shard, chunk; a rank without a diagonal block starts at stage 1), in
// the backward the same blocks at the same stages as in the forward.  Inputs
// come one stage ahead directly from their owner (K/V of chunk c from rank c,
// Q -- and in the backward dO with its row statistics -- of shard r from rank
// r) into slot t % 2 of the receiver's double-buffered receive slots; a result
// that belongs to another rank (a transferred block's partial O or dQ, a ring
// block's dK/dV) is written to result slot t % 2 and sent one stage later.
// Within a stage the sends and receives come first (all of them form one
// batched point-to-point group), then the computation, then the merge.
#include <algorithm>
#include <vector>

#include "hsap_internal.h"

using namespace hsap;

namespace {

struct Block {
  int32_t r, c;
};

// The blocks of every rank in stage order, each rank's first compute stage, the number of stages
// after the last compute stage (S: the last stage returns results and merges), and the part
// indices: part[r * P + c] = rank of chunk c among the chunks with a block of shard r, kpart[c * P
// + r] = rank of shard r among the shards with a block in chunk c.
struct Layout {
  int32_t P = 0, S = 0;
  std::vector<std::vector<Block>> blocks;
  std::vector<int32_t> first, part, parts, kpart, kparts;
};

hsap_status layout_blocks(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank,
                          const int64_t* rank_offsets, const int32_t* num_stages, int64_t capacity, Layout* L) {
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
  L->P = P;
  L->blocks.assign((size_t)P, {});
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c)
      if (block_tiles[(int64_t)r * P + c] > 0) L->blocks[(size_t)exec_rank[(int64_t)r * P + c]].push_back(Block{r, c});
  auto ring_step = [P](const Block& b) { return ((b.r - b.c) % P + P) % P; };
  for (auto& list : L->blocks)
    std::sort(list.begin(), list.end(), [&](const Block& a, const Block& b) {
      const int da = a.r == a.c ? 0 : 1, db = b.r == b.c ? 0 : 1;
      if (da != db) return da < db;
      if (ring_step(a) != ring_step(b)) return ring_step(a) < ring_step(b);
      if (a.r != b.r) return a.r < b.r;
      return a.c < b.c;
    });
  // a rank without a diagonal block starts at stage 1: its first input has to arrive first
  L->first.assign((size_t)P, 0);
  L->S = 0;
  for (int32_t e = 0; e < P; ++e) {
    const auto& list = L->blocks[(size_t)e];
    L->first[(size_t)e] = !list.empty() && list[0].r == list[0].c ? 0 : 1;
    L->S = std::max<int32_t>(L->S, L->first[(size_t)e] + (int32_t)list.size());
  }
  L->part.assign((size_t)P * P, -1);
  L->parts.assign((size_t)P, 0);
  L->kpart.assign((size_t)P * P, -1);
  L->kparts.assign((size_t)P, 0);
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c)
      if (block_tiles[(int64_t)r * P + c] > 0) L->part[(size_t)r * P + c] = L->parts[(size_t)r]++;
  for (int32_t c = 0; c < P; ++c)
    for (int32_t r = 0; r < P; ++r)
      if (block_tiles[(int64_t)r * P + c] > 0) L->kpart[(size_t)c * P + r] = L->kparts[(size_t)c]++;
  return HSAP_OK;
}

// Writes the per-(rank, stage) communication (sorted by peer, send before receive, tensor, shard,
// chunk), computation and merges into ops in rank order; the two-call capacity protocol.
hsap_status write_program(const Layout& L, std::vector<std::vector<hsap_op>>& comm,
                          const std::vector<std::vector<hsap_op>>& comp, const std::vector<std::vector<hsap_op>>& merge,
                          hsap_op* ops, int64_t capacity, int64_t* rank_offsets, int32_t* num_stages) {
  const int32_t P = L.P, S = L.S;
  int64_t count = 0;
  for (int32_t e = 0; e < P; ++e) {
    rank_offsets[e] = count;
    for (int32_t t = 0; t <= S; ++t) {
      const size_t i = (size_t)e * (S + 1) + t;
      auto& cm = comm[i];
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
      for (const auto& o : comp[i]) emit(o);
      for (const auto& o : merge[i]) emit(o);
    }
  }
  rank_offsets[P] = count;
  *num_stages = S + 1;
  if (!ops || count > capacity)
    HSAP_FAIL(HSAP_ERR_CAPACITY, "program needs %lld ops, capacity %lld", (long long)count, (long long)capacity);
  return HSAP_OK;
}

}  // namespace

extern "C" hsap_status hsap_emit_forward(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank,
                                         hsap_op* ops, int64_t capacity, int64_t* rank_offsets,
                                         int32_t* num_stages) {
  clear_error();
  Layout lay;
  const hsap_status st = layout_blocks(sp_degree, block_tiles, exec_rank, rank_offsets, num_stages, capacity, &lay);
  if (st != HSAP_OK) return st;
  const int32_t P = lay.P, S = lay.S;
  const auto& blocks = lay.blocks;
  const auto& first = lay.first;
  const auto& part = lay.part;
  const auto& parts = lay.parts;

  // ops per (rank, stage): communication, computation and merges separately
  const size_t cells = (size_t)P * (S + 1);
  std::vector<std::vector<hsap_op>> comm(cells), comp(cells), merge(cells);
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
  for (int32_t e = 0; e < P; ++e)
    if (parts[(size_t)e] > 0) merge[at(e, S)].push_back(hsap_op{HSAP_OP_MERGE, HSAP_T_NONE, -1, S, e, -1, -1, parts[(size_t)e]});
  return write_program(lay, comm, comp, merge, ops, capacity, rank_offsets, num_stages);
}

// The backward: the forward's blocks on the same ranks at the same stages.  A ring block (r, c)
// on rank r needs chunk c's K/V (from rank c, one stage ahead) and returns its dK/dV part to rank
// c a stage later; a transferred block (r, c) on rank c needs shard r's Q and dO (with the row
// statistics, from rank r, one stage ahead) and returns its dQ part to rank r a stage later.  The
// part that stays is written locally: dQ part part(r, c) of the own shard, dK/dV part kpart(c, r)
// of the own chunk (a diagonal block writes both).  In the last stage each rank sums its dQ parts
// in part order (MERGE of tensor DQ) and its dK/dV parts likewise (MERGE of tensor DKV).
extern "C" hsap_status hsap_emit_backward(int32_t sp_degree, const int64_t* block_tiles, const int32_t* exec_rank,
                                          hsap_op* ops, int64_t capacity, int64_t* rank_offsets,
                                          int32_t* num_stages) {
  clear_error();
  Layout lay;
  const hsap_status st = layout_blocks(sp_degree, block_tiles, exec_rank, rank_offsets, num_stages, capacity, &lay);
  if (st != HSAP_OK) return st;
  const int32_t P = lay.P, S = lay.S;
  const size_t cells = (size_t)P * (S + 1);
  std::vector<std::vector<hsap_op>> comm(cells), comp(cells), merge(cells);
  auto at = [&](int32_t e, int32_t t) { return (size_t)e * (S + 1) + t; };
  for (int32_t e = 0; e < P; ++e)
    for (int32_t i = 0; i < (int32_t)lay.blocks[(size_t)e].size(); ++i) {
      const Block b = lay.blocks[(size_t)e][(size_t)i];
      const int32_t t = lay.first[(size_t)e] + i;
      int32_t in_slot = -1, out_slot = -1;
      if (b.r == e && b.c != e) {  // ring block: K/V in, dK/dV back to the chunk's owner
        comm[at(b.c, t - 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_KV, e, t - 1, -1, b.c, -1, -1});
        comm[at(e, t - 1)].push_back(hsap_op{HSAP_OP_RECV, HSAP_T_KV, b.c, t - 1, -1, b.c, -1, t % 2});
        comm[at(e, t + 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_DKV, b.c, t + 1, b.r, b.c, t % 2, -1});
        comm[at(b.c, t + 1)].push_back(
            hsap_op{HSAP_OP_RECV, HSAP_T_DKV, e, t + 1, b.r, b.c, -1, lay.kpart[(size_t)b.c * P + b.r]});
        in_slot = out_slot = t % 2;
      } else if (b.c == e && b.r != e) {  // transferred block: Q and dO in, dQ back to the shard's owner
        for (int32_t tensor : {HSAP_T_Q, HSAP_T_DO}) {
          comm[at(b.r, t - 1)].push_back(hsap_op{HSAP_OP_SEND, tensor, e, t - 1, b.r, -1, -1, -1});
          comm[at(e, t - 1)].push_back(hsap_op{HSAP_OP_RECV, tensor, b.r, t - 1, b.r, -1, -1, t % 2});
        }
        comm[at(e, t + 1)].push_back(hsap_op{HSAP_OP_SEND, HSAP_T_DQ, b.r, t + 1, b.r, b.c, t % 2, -1});
        comm[at(b.r, t + 1)].push_back(
            hsap_op{HSAP_OP_RECV, HSAP_T_DQ, e, t + 1, b.r, b.c, -1, lay.part[(size_t)b.r * P + b.c]});
        in_slot = out_slot = t % 2;
      }
      comp[at(e, t)].push_back(hsap_op{HSAP_OP_COMPUTE, HSAP_T_NONE, -1, t, b.r, b.c, in_slot, out_slot});
    }
  for (int32_t e = 0; e < P; ++e) {
    if (lay.parts[(size_t)e] > 0)
      merge[at(e, S)].push_back(hsap_op{HSAP_OP_MERGE, HSAP_T_DQ, -1, S, e, -1, -1, lay.parts[(size_t)e]});
    if (lay.kparts[(size_t)e] > 0)
      merge[at(e, S)].push_back(hsap_op{HSAP_OP_MERGE, HSAP_T_DKV, -1, S, -1, e, -1, lay.kparts[(size_t)e]});
  }
  return write_program(lay, comm, comp, merge, ops, capacity, rank_offsets, num_stages);
}
