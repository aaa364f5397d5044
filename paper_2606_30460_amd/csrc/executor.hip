// Step executor: plans each packed batch on the host, uploads every list with
// one asynchronous copy from pinned memory, and runs one shard's forward and
// backward with one call each.  Host code only; the work is done by the entry
// points of the other translation units.
#include <algorithm>
#include <cstring>
#include <vector>

#include "hsap_internal.h"

using namespace hsap;

namespace {

// Pinned staging buffers for the list uploads, used in a ring.  The host may rewrite a buffer only
// once the copy out of it has run; an event tells it so, but an event marker costs the stream a
// gap of several microseconds, so one is recorded only after every kEventEvery-th upload: before
// rewriting the buffer of upload u - kStaging, the host waits for the first event recorded at or
// after that upload (the stream runs in order).  kEventEvery <= kStaging keeps that event in the
// past.
constexpr int kStaging = 16;
constexpr int kEventEvery = 8;
static_assert(kEventEvery <= kStaging, "the awaited event must precede the upload that waits");

// Device or pinned allocation that grows (never shrinks) to the largest size asked for.
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

// Words (int32) of a list section rounded up to 16 bytes.
inline size_t words16(size_t words) { return (words + 3) & ~size_t(3); }

}  // namespace

struct hsap_executor {
  hsap_attn_desc desc;
  Geom geom;
  int32_t options = 0;
  int32_t max_run_tiles = -1;
  int32_t resident_workgroups = 0;
  int device = 0;
  int64_t nq = 0, nk = 0;

  // host planner output (pageable)
  std::vector<hsap_tile> tiles, sorted_q, sorted_k, sorted_all;
  std::vector<hsap_run> runs_q, runs_k, runs_all;
  std::vector<int64_t> step_offsets, pairs;
  std::vector<int32_t> slot_map;
  std::vector<uint8_t> final_tile;  // per q-tile: 1 when its only part is written final by the partial forward
  std::vector<int32_t> merged_tiles;  // the other q-tiles, in order: the merge's rows
  std::vector<int32_t> zero_ktiles;   // k-tiles (c * nk + k_tile) of chunks with tiles that no query reaches

  // pinned staging ring; upload u uses pinned[u % kStaging], and when u % kEventEvery is
  // kEventEvery - 1 an event recorded after its copy sits in uploaded[u % kStaging]
  DevBuf pinned[kStaging];
  hipEvent_t uploaded[kStaging] = {};
  int64_t event_upload[kStaging];  // the upload each event follows (-1: none yet)
  int64_t uploads = 0;             // uploads issued so far

  // device side
  DevBuf lists;  // [sorted_q | runs_q | sorted_k | runs_k | sorted_all | runs_all | cu | merged_tiles | zero_ktiles]
  int32_t* doc_start = nullptr;  // start(t) per position, for the backward only
  DevBuf o_part, lse_part;
  float* delta = nullptr;

  // current plan
  bool planned = false;
  hsap_exec_info info{};
  const hsap_tile* d_tiles_q = nullptr;
  const hsap_run* d_runs_q = nullptr;
  const hsap_tile* d_tiles_k = nullptr;
  const hsap_run* d_runs_k = nullptr;
  const hsap_tile* d_tiles_all = nullptr;
  const hsap_run* d_runs_all = nullptr;
  const int32_t* d_merged_tiles = nullptr;
  const int32_t* d_zero_ktiles = nullptr;
  const int32_t* d_cu = nullptr;  // the plan's cu_seqlens (the forwards search it for document starts)
  int32_t num_docs = 0;
  std::vector<uint8_t> chunk_has_tiles;
};

namespace {

hsap_status hip_fail(const char* what, hipError_t e) {
  HSAP_FAIL(HSAP_ERR_HIP, "executor: %s: %s", what, hipGetErrorString(e));
}

// Grow a device buffer; the stream is synchronised first so no queued kernel still reads the old one.
hsap_status grow_device(DevBuf& b, size_t bytes, hipStream_t stream) {
  if (bytes <= b.bytes) return HSAP_OK;
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail("stream synchronize", e);
  const size_t want = std::max(bytes, b.bytes + b.bytes / 2);
  if (b.p) hipFree(b.p);
  b.p = nullptr;
  b.bytes = 0;
  e = hipMalloc(&b.p, want);
  if (e != hipSuccess) {
    b.p = nullptr;
    return hip_fail("device allocation", e);
  }
  b.bytes = want;
  return HSAP_OK;
}

// Grow a pinned staging buffer whose previous upload has completed.
hsap_status grow_pinned(DevBuf& b, size_t bytes) {
  if (bytes <= b.bytes) return HSAP_OK;
  if (b.p) hipHostFree(b.p);
  b.p = nullptr;
  b.bytes = 0;
  const size_t want = std::max(bytes, size_t(4096));
  const hipError_t e = hipHostMalloc(&b.p, want, hipHostMallocDefault);
  if (e != hipSuccess) {
    b.p = nullptr;
    return hip_fail("pinned allocation", e);
  }
  b.bytes = want;
  return HSAP_OK;
}

void release(hsap_executor* ex) {
  for (int i = 0; i < kStaging; ++i) {
    if (ex->pinned[i].p) hipHostFree(ex->pinned[i].p);
    if (ex->uploaded[i]) hipEventDestroy(ex->uploaded[i]);
  }
  void* dev[] = {ex->lists.p, ex->doc_start, ex->o_part.p, ex->lse_part.p, ex->delta};
  for (void* p : dev)
    if (p) hipFree(p);
  delete ex;
}

// hsap_plan_runs with a growing run vector (two-call pattern only when it is too small)
hsap_status runs_for(const hsap_executor* ex, int32_t major, int32_t split, std::vector<hsap_tile>& sorted,
                     std::vector<hsap_run>& runs, int64_t* num_runs, int32_t* num_slots) {
  const int64_t T = ex->info.num_tiles;
  sorted.resize((size_t)std::max<int64_t>(T, 1));
  if (runs.empty()) runs.resize(64);
  hsap_status st = hsap_plan_runs(&ex->desc.shard, ex->tiles.data(), T, major, split, sorted.data(), runs.data(),
                                  (int64_t)runs.size(), num_runs, num_slots);
  if (st == HSAP_ERR_CAPACITY) {
    runs.resize((size_t)*num_runs);
    st = hsap_plan_runs(&ex->desc.shard, ex->tiles.data(), T, major, split, sorted.data(), runs.data(),
                        (int64_t)runs.size(), num_runs, num_slots);
  }
  return st;
}

}  // namespace

extern "C" {

hsap_status hsap_executor_create(const hsap_attn_desc* desc, int32_t options, int32_t max_run_tiles,
                                 hsap_executor** out) {
  clear_error();
  if (!out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  Geom g;
  const hsap_status st = check_attn(desc, &g);
  if (st != HSAP_OK) return st;
  if (options & ~(HSAP_EXEC_BACKWARD | HSAP_EXEC_FUSED)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "unknown option bits %#x", options);
  if (max_run_tiles < -1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "max_run_tiles %d < -1", max_run_tiles);
  if (desc->shard.sp_degree > HSAP_MAX_MERGE_PARTS)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "sp_degree %d above the merge limit %d", desc->shard.sp_degree,
              HSAP_MAX_MERGE_PARTS);
  if ((options & HSAP_EXEC_BACKWARD) && !backward_supported(desc))
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no backward kernel for head_dim=%d BM=%d BN=%d", desc->head_dim,
              desc->shard.block_m, desc->shard.block_n);

  hsap_executor* ex = new hsap_executor();
  ex->desc = *desc;
  ex->geom = g;
  ex->options = options;
  ex->max_run_tiles = max_run_tiles;
  ex->nq = g.n / desc->shard.block_m;
  ex->nk = g.n / desc->shard.block_n;
  ex->step_offsets.assign((size_t)g.P + 1, 0);
  ex->pairs.assign((size_t)g.P, 0);
  ex->chunk_has_tiles.assign((size_t)g.P, 0);
  int cus = 0;
  hipError_t e = hipGetDevice(&ex->device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, ex->device);
  for (int i = 0; i < kStaging; ++i) ex->event_upload[i] = -1;
  for (int i = 0; e == hipSuccess && i < kStaging; ++i)
    e = hipEventCreateWithFlags(&ex->uploaded[i], hipEventDisableTiming);
  if (e == hipSuccess && (options & HSAP_EXEC_BACKWARD))
    e = hipMalloc((void**)&ex->doc_start, (size_t)g.N * sizeof(int32_t));
  if (e == hipSuccess && (options & HSAP_EXEC_BACKWARD))
    e = hipMalloc((void**)&ex->delta, (size_t)g.n * desc->heads_q * sizeof(float));
  if (e != hipSuccess) {
    release(ex);
    return hip_fail("create", e);
  }
  ex->resident_workgroups = std::max(1, fwd_resident_per_cu(desc)) * std::max(cus, 1);
  *out = ex;
  return HSAP_OK;
}

void hsap_executor_destroy(hsap_executor* ex) {
  if (!ex) return;
  const int own = ex->device;
  int cur = own;
  if (hipGetDevice(&cur) == hipSuccess && cur != own) hipSetDevice(own);
  hipDeviceSynchronize();
  release(ex);
  if (cur != own) hipSetDevice(cur);
}

hsap_status hsap_executor_plan(hsap_executor* ex, const int32_t* cu_seqlens, int32_t num_docs, void* hip_stream) {
  clear_error();
  if (!ex || !cu_seqlens) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor or cu_seqlens");
  const hipStream_t stream = (hipStream_t)hip_stream;
  const hsap_shard_desc& sd = ex->desc.shard;
  const int32_t P = sd.sp_degree;
  ex->planned = false;

  // 1. tiles (the planner validates cu_seqlens and the geometry)
  int64_t T = 0;
  if (ex->tiles.empty()) ex->tiles.resize(256);
  hsap_status st = hsap_plan(cu_seqlens, num_docs, &sd, ex->tiles.data(), (int64_t)ex->tiles.size(), &T,
                             ex->step_offsets.data(), ex->pairs.data());
  if (st == HSAP_ERR_CAPACITY) {
    ex->tiles.resize((size_t)T);
    st = hsap_plan(cu_seqlens, num_docs, &sd, ex->tiles.data(), (int64_t)ex->tiles.size(), &T,
                   ex->step_offsets.data(), ex->pairs.data());
  }
  if (st != HSAP_OK) return st;
  hsap_exec_info info{};
  info.num_tiles = T;
  for (int64_t i = 0; i < T; ++i) info.num_full_tiles += ex->tiles[(size_t)i].kind == HSAP_TILE_FULL;
  for (int32_t s = 0; s < P; ++s) info.useful_pairs += ex->pairs[(size_t)s];
  ex->info = info;

  // 2. q-major runs, split as configured; slots renumbered densely
  int32_t split = ex->max_run_tiles;
  if (split < 0) split = hsap_split_length(&sd, T, ex->desc.heads_q, ex->resident_workgroups);
  if (split < 0) return HSAP_ERR_INVALID_ARG;
  int64_t RQ = 0;
  int32_t slots = 0;
  st = runs_for(ex, HSAP_MAJOR_Q, split, ex->sorted_q, ex->runs_q, &RQ, &slots);
  if (st != HSAP_OK) return st;
  ex->slot_map.assign((size_t)slots, -1);
  for (int64_t i = 0; i < RQ; ++i) ex->slot_map[(size_t)ex->runs_q[(size_t)i].slot] = 1;
  int32_t parts = 0;
  for (auto& m : ex->slot_map) m = m < 0 ? -1 : parts++;
  if (parts > HSAP_MAX_MERGE_PARTS && split > 0) {  // too many pieces to merge in one call: plan without split
    split = 0;
    st = runs_for(ex, HSAP_MAJOR_Q, 0, ex->sorted_q, ex->runs_q, &RQ, &slots);
    if (st != HSAP_OK) return st;
    ex->slot_map.assign((size_t)slots, -1);
    for (int64_t i = 0; i < RQ; ++i) ex->slot_map[(size_t)ex->runs_q[(size_t)i].slot] = 1;
    parts = 0;
    for (auto& m : ex->slot_map) m = m < 0 ? -1 : parts++;
  }
  std::fill(ex->chunk_has_tiles.begin(), ex->chunk_has_tiles.end(), 0);
  for (int32_t s = 0; s < slots; ++s)
    if (ex->slot_map[(size_t)s] >= 0) ex->chunk_has_tiles[(size_t)(s % P)] = 1;
  for (int64_t i = 0; i < RQ; ++i) ex->runs_q[(size_t)i].slot = ex->slot_map[(size_t)ex->runs_q[(size_t)i].slot];
  // A q-tile with exactly one run holding tiles (one chunk, unsplit) has a single part: the merge
  // would return it unchanged, so that run writes the final output and the merge skips the
  // q-tile; the q-tile's empty runs (LSE = -inf parts nobody reads) are dropped.
  {
    std::vector<int32_t> busy((size_t)ex->nq, 0);
    for (int64_t i = 0; i < RQ; ++i)
      if (ex->runs_q[(size_t)i].count > 0) ++busy[(size_t)ex->runs_q[(size_t)i].tile];
    ex->final_tile.assign((size_t)ex->nq, 0);
    int64_t kept = 0;
    for (int64_t i = 0; i < RQ; ++i) {
      hsap_run r = ex->runs_q[(size_t)i];
      if (busy[(size_t)r.tile] == 1) {
        if (r.count == 0) continue;
        r.slot = kFinalSlot;
        ex->final_tile[(size_t)r.tile] = 1;
      }
      ex->runs_q[(size_t)kept++] = r;
    }
    RQ = kept;
  }
  ex->info.num_runs_q = RQ;
  ex->info.num_parts = parts;
  ex->info.final_q_tiles = 0;
  ex->merged_tiles.clear();
  for (int64_t t = 0; t < ex->nq; ++t) {
    if (ex->final_tile[(size_t)t]) ++ex->info.final_q_tiles;
    else ex->merged_tiles.push_back((int32_t)t);
  }
  ex->info.split_length = split;
  for (int32_t c = 0; c < P; ++c)
    if (ex->chunk_has_tiles[(size_t)c]) {
      ++ex->info.chunks_with_tiles;
      ex->info.chunk_mask |= 1ull << c;
    }

  // 3. k-major and fused runs
  int64_t RK = 0, RA = 0;
  if (ex->options & HSAP_EXEC_BACKWARD) {
    st = runs_for(ex, HSAP_MAJOR_K, 0, ex->sorted_k, ex->runs_k, &RK, nullptr);
    if (st != HSAP_OK) return st;
  }
  if (ex->options & (HSAP_EXEC_FUSED | HSAP_EXEC_BACKWARD)) {  // fused forward and the backward's dQ
    st = runs_for(ex, HSAP_MAJOR_Q_ALL, 0, ex->sorted_all, ex->runs_all, &RA, nullptr);
    if (st != HSAP_OK) return st;
  }
  ex->info.num_runs_k = RK;
  ex->info.num_runs_all = RA;
  // dK/dV rows of a chunk with tiles are written by the k-major run of their k-tile; the k-tiles
  // without one (no query of the shard reaches them) are zeroed by the backward instead
  ex->zero_ktiles.clear();
  if (RK) {
    const int64_t nk = ex->geom.n / sd.block_n;
    std::vector<uint8_t> reached((size_t)P * nk, 0);
    for (int64_t i = 0; i < RK; ++i) reached[(size_t)(ex->runs_k[(size_t)i].slot * nk + ex->runs_k[(size_t)i].tile)] = 1;
    for (int32_t c = 0; c < P; ++c)
      if (ex->chunk_has_tiles[(size_t)c])
        for (int64_t t = 0; t < nk; ++t)
          if (!reached[(size_t)(c * nk + t)]) ex->zero_ktiles.push_back((int32_t)(c * nk + t));
  }

  // 4. partial workspace for this plan's parts
  const size_t part_rows = (size_t)ex->geom.n * ex->desc.heads_q;
  st = grow_device(ex->o_part, (size_t)parts * part_rows * ex->desc.head_dim * sizeof(float), stream);
  if (st == HSAP_OK) st = grow_device(ex->lse_part, (size_t)parts * part_rows * sizeof(float), stream);
  if (st != HSAP_OK) return st;

  // 5. one staging buffer, one upload
  const size_t w_tq = words16((size_t)T * 4), w_rq = words16((size_t)RQ * 4);
  const size_t w_tk = RK ? w_tq : 0, w_rk = words16((size_t)RK * 4);
  const size_t w_ta = RA ? w_tq : 0, w_ra = words16((size_t)RA * 4);
  const size_t w_cu = words16((size_t)num_docs + 1);
  const size_t w_mt = words16(ex->merged_tiles.size()), w_zt = words16(ex->zero_ktiles.size());
  const size_t o_rq = w_tq, o_tk = o_rq + w_rq, o_rk = o_tk + w_tk, o_ta = o_rk + w_rk, o_ra = o_ta + w_ta,
               o_cu = o_ra + w_ra, o_mt = o_cu + w_cu, o_zt = o_mt + w_mt, words = o_zt + w_zt;
  const int64_t u = ex->uploads;
  const int slot = (int)(u % kStaging);
  if (u >= kStaging) {  // the buffer last served upload u - kStaging
    const int64_t prev = u - kStaging, ev = prev + (kEventEvery - 1 - prev % kEventEvery);
    if (ex->event_upload[ev % kStaging] != ev) HSAP_FAIL(HSAP_ERR_HIP, "executor: staging event bookkeeping");
    const hipError_t e = hipEventSynchronize(ex->uploaded[ev % kStaging]);
    if (e != hipSuccess) return hip_fail("staging wait", e);
  }
  st = grow_pinned(ex->pinned[slot], words * 4);
  if (st == HSAP_OK) st = grow_device(ex->lists, words * 4, stream);
  if (st != HSAP_OK) return st;
  int32_t* h = (int32_t*)ex->pinned[slot].p;
  std::memcpy(h, ex->sorted_q.data(), (size_t)T * sizeof(hsap_tile));
  std::memcpy(h + o_rq, ex->runs_q.data(), (size_t)RQ * sizeof(hsap_run));
  if (RK) {
    std::memcpy(h + o_tk, ex->sorted_k.data(), (size_t)T * sizeof(hsap_tile));
    std::memcpy(h + o_rk, ex->runs_k.data(), (size_t)RK * sizeof(hsap_run));
  }
  if (RA) {
    std::memcpy(h + o_ta, ex->sorted_all.data(), (size_t)T * sizeof(hsap_tile));
    std::memcpy(h + o_ra, ex->runs_all.data(), (size_t)RA * sizeof(hsap_run));
  }
  std::memcpy(h + o_cu, cu_seqlens, ((size_t)num_docs + 1) * sizeof(int32_t));
  std::memcpy(h + o_mt, ex->merged_tiles.data(), ex->merged_tiles.size() * sizeof(int32_t));
  std::memcpy(h + o_zt, ex->zero_ktiles.data(), ex->zero_ktiles.size() * sizeof(int32_t));
  hipError_t e = hipMemcpyAsync(ex->lists.p, h, words * 4, hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail("list upload", e);
  if (u % kEventEvery == kEventEvery - 1) {
    e = hipEventRecord(ex->uploaded[slot], stream);
    if (e != hipSuccess) return hip_fail("event record", e);
    ex->event_upload[slot] = u;
  }
  ex->uploads = u + 1;

  int32_t* d = (int32_t*)ex->lists.p;
  ex->d_tiles_q = (const hsap_tile*)d;
  ex->d_runs_q = (const hsap_run*)(d + o_rq);
  ex->d_tiles_k = RK ? (const hsap_tile*)(d + o_tk) : nullptr;
  ex->d_runs_k = RK ? (const hsap_run*)(d + o_rk) : nullptr;
  ex->d_tiles_all = RA ? (const hsap_tile*)(d + o_ta) : nullptr;
  ex->d_runs_all = RA ? (const hsap_run*)(d + o_ra) : nullptr;
  ex->d_merged_tiles = d + o_mt;
  ex->d_zero_ktiles = d + o_zt;
  ex->d_cu = d + o_cu;
  ex->num_docs = num_docs;

  // 6. start(t) for every position, read by the backward's masks (the forwards search cu_seqlens)
  if (ex->options & HSAP_EXEC_BACKWARD) {
    st = hsap_doc_start(d + o_cu, num_docs, ex->geom.N, ex->doc_start, hip_stream);
    if (st != HSAP_OK) return st;
  }
  ex->planned = true;
  return HSAP_OK;
}

hsap_status hsap_executor_info(const hsap_executor* ex, hsap_exec_info* info) {
  clear_error();
  if (!ex || !info) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor or info");
  if (!ex->planned) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "executor has no plan");
  *info = ex->info;
  return HSAP_OK;
}

hsap_status hsap_executor_partial_forward(hsap_executor* ex, const void* q, const void* k, const void* v,
                                          void* o_out, float* lse_out, void* hip_stream) {
  clear_error();
  if (!ex) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor");
  if (!ex->planned) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "executor has no plan");
  if (!q || !k || !v || !o_out || !lse_out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  return executor_forward(&ex->desc, false, q, k, v, ex->d_cu, ex->num_docs, ex->d_tiles_q, ex->d_runs_q,
                          ex->info.num_runs_q, (float*)ex->o_part.p, (float*)ex->lse_part.p, ex->info.num_parts,
                          o_out, lse_out, (hipStream_t)hip_stream);
}

hsap_status hsap_executor_merge(hsap_executor* ex, void* o_out, float* lse_out, void* hip_stream) {
  clear_error();
  if (!ex) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor");
  if (!ex->planned) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "executor has no plan");
  if (!o_out || !lse_out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  const int32_t parts = ex->info.num_parts;
  const size_t rows = (size_t)ex->geom.n * ex->desc.heads_q;
  const float* o_ptrs[HSAP_MAX_MERGE_PARTS];
  const float* l_ptrs[HSAP_MAX_MERGE_PARTS];
  for (int32_t p = 0; p < parts; ++p) {
    o_ptrs[p] = (const float*)ex->o_part.p + (size_t)p * rows * ex->desc.head_dim;
    l_ptrs[p] = (const float*)ex->lse_part.p + (size_t)p * rows;
  }
  if (ex->info.final_q_tiles == ex->nq) return HSAP_OK;  // every q-tile was written final
  return lse_merge(parts, o_ptrs, l_ptrs, ex->geom.n, ex->desc.heads_q, ex->desc.head_dim, o_out, lse_out,
                   ex->d_merged_tiles, (int32_t)ex->merged_tiles.size(), ex->desc.shard.block_m,
                   (hipStream_t)hip_stream);
}

hsap_status hsap_executor_forward(hsap_executor* ex, const void* q, const void* k, const void* v, int32_t fused,
                                  void* o_out, float* lse_out, void* hip_stream) {
  clear_error();
  if (!ex) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor");
  if (!ex->planned) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "executor has no plan");
  if (!q || !k || !v || !o_out || !lse_out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (fused) {
    if (!(ex->options & HSAP_EXEC_FUSED)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "fused forward needs HSAP_EXEC_FUSED");
    return executor_forward(&ex->desc, true, q, k, v, ex->d_cu, ex->num_docs, ex->d_tiles_all, ex->d_runs_all,
                            ex->info.num_runs_all, nullptr, nullptr, 0, o_out, lse_out, (hipStream_t)hip_stream);
  }
  const hsap_status st = hsap_executor_partial_forward(ex, q, k, v, o_out, lse_out, hip_stream);
  if (st != HSAP_OK) return st;
  return hsap_executor_merge(ex, o_out, lse_out, hip_stream);
}

hsap_status hsap_executor_backward(hsap_executor* ex, const void* q, const void* k, const void* v, const void* d_o,
                                   const void* o, const float* lse, void* dq, void* dk, void* dv, void* hip_stream) {
  clear_error();
  if (!ex) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL executor");
  if (!(ex->options & HSAP_EXEC_BACKWARD)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "backward needs HSAP_EXEC_BACKWARD");
  if (!ex->planned) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "executor has no plan");
  if (!q || !k || !v || !d_o || !o || !lse || !dq || !dk || !dv)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  const hipStream_t stream = (hipStream_t)hip_stream;
  const int64_t d = ex->desc.head_dim;
  // in a chunk with tiles, dK/dV rows of k-tiles that no query reaches have no owning run: zeroed
  // here (the listed k-tiles only; the kernels write every other row of those chunks)
  const int64_t ktile_bytes = (int64_t)ex->desc.shard.block_n * ex->desc.heads_kv * d * 2;
  hsap_status st = zero_tiles(dk, dv, ex->d_zero_ktiles, (int32_t)ex->zero_ktiles.size(), ktile_bytes, stream);
  // the preprocess (delta = rowsum(dO o O)) runs inside the dQ kernel, which reads dO anyway
  if (st == HSAP_OK)
    st = attn_bwd_bf16_delta(&ex->desc, q, k, v, d_o, o, lse, ex->delta, ex->doc_start, ex->d_tiles_k, ex->d_runs_k,
                             ex->info.num_runs_k, ex->d_tiles_all, ex->d_runs_all, ex->info.num_runs_all, dq, dk, dv,
                             stream);
  return st;
}

}  // extern "C"
