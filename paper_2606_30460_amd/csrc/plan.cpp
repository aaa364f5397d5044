// Host side of libhsap: argument checks, error strings and the tile planner.
//
// The planner follows compile step 1 of the SAP section: the packed causal
// mask is cut into blocks that one rank computes against one K/V chunk and
// each block is classified by its attention pattern, so blocks with nothing
// to attend are neither transferred nor computed.  Here the blocks are
// BM x BN tiles and the classes are EMPTY (dropped), FULL and MASKED.
//
// Counting is interval arithmetic, never pair by pair:
//   * a q-tile covers consecutive global positions [qa, qb] (tiles never
//     straddle two zigzag pieces), so the keys its rows may attend form the
//     single window [start(qa), qb]; every k-tile meeting that window holds
//     at least one allowed pair and every other k-tile holds none;
//   * a tile is FULL iff start(qb) <= ka and kb <= qa (the latest document
//     start among its rows is at or before its first key, and its last key is
//     at or before its first query);
//   * otherwise its pair count is summed per document segment of its rows as
//     two arithmetic series (rows before the k-tile's end, rows after it).
#include <algorithm>
#include <cstdarg>
#include <cstring>
#include <numeric>
#include <vector>

#include "hsap_internal.h"

namespace hsap {

static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
}

void clear_error() { g_last_error.clear(); }

hsap_status check_shard(const hsap_shard_desc* d, Geom* g) {
  if (!d) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "shard descriptor is NULL");
  const int32_t B = d->batch <= 0 ? 1 : d->batch;
  if (d->batch < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "batch %d < 0", d->batch);
  if (d->total_tokens <= 0 || d->total_tokens * B > INT32_MAX)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "total_tokens %lld x batch %d outside 1..2^31-1", (long long)d->total_tokens, B);
  if (d->sp_degree < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "sp_degree %d < 1", d->sp_degree);
  if (d->shard_id < 0 || d->shard_id >= d->sp_degree)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "shard_id %d outside 0..%d", d->shard_id, d->sp_degree - 1);
  if (d->layout != HSAP_LAYOUT_CONTIGUOUS && d->layout != HSAP_LAYOUT_ZIGZAG)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "unknown layout %d", d->layout);
  const int64_t N = d->total_tokens, P = d->sp_degree;
  const int64_t split = d->layout == HSAP_LAYOUT_ZIGZAG ? 2 * P : P;
  if (N % split)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "total_tokens %lld not divisible by %lld", (long long)N, (long long)split);
  const int64_t piece = N / split;
  if (d->block_m <= 0 || d->block_n <= 0)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "tile sizes must be positive (BM=%d BN=%d)", d->block_m, d->block_n);
  if (piece % d->block_m || piece % d->block_n)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "BM=%d and BN=%d must divide the %s length %lld", d->block_m, d->block_n,
              d->layout == HSAP_LAYOUT_ZIGZAG ? "zigzag piece" : "shard", (long long)piece);
  g->Ns = N;
  g->ns = N / P;
  g->N = N * B;
  g->n = (N / P) * B;
  g->m = piece;
  g->P = (int32_t)P;
  g->layout = d->layout;
  g->B = B;
  return HSAP_OK;
}

hsap_status check_attn(const hsap_attn_desc* d, Geom* g) {
  if (!d) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "attention descriptor is NULL");
  hsap_status st = check_shard(&d->shard, g);
  if (st != HSAP_OK) return st;
  if (d->heads_q <= 0 || d->heads_kv <= 0 || d->heads_q % d->heads_kv)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "heads_q=%d must be a positive multiple of heads_kv=%d", d->heads_q,
              d->heads_kv);
  if (!(d->softmax_scale > 0.f) || d->softmax_scale > 1e30f)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
  if (d->head_dim != 64 && d->head_dim != 128)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d->head_dim);
  return HSAP_OK;
}

namespace {

// Positions of shard x's local rows, as (global start, local start, length) pieces, one or two
// per sequence of the batch; piece i belongs to sequence i / (pieces per sequence).
struct Piece {
  int64_t global0, local0, len;
};

int pieces_per_sequence(const Geom& g) { return g.layout == HSAP_LAYOUT_CONTIGUOUS ? 1 : 2; }

void shard_pieces(const Geom& g, int32_t x, std::vector<Piece>& out) {
  out.clear();
  for (int32_t b = 0; b < g.B; ++b) {
    const int64_t gb = (int64_t)b * g.Ns, lb = (int64_t)b * g.ns;
    if (g.layout == HSAP_LAYOUT_CONTIGUOUS) {
      out.push_back({gb + (int64_t)x * g.ns, lb, g.ns});
    } else {
      out.push_back({gb + (int64_t)x * g.m, lb, g.m});
      out.push_back({gb + (int64_t)(2 * g.P - 1 - x) * g.m, lb + g.m, g.m});
    }
  }
}

// Index of the document holding position t (the last k with cu[k] <= t).
inline int64_t doc_of(const int32_t* cu, int32_t num_docs, int64_t t) {
  const int32_t* it = std::upper_bound(cu, cu + num_docs + 1, (int32_t)t);
  return (int64_t)(it - cu) - 1;
}

// Allowed pairs between query rows [qa, qb] (document of qa: dq) and keys [ka, kb].
int64_t tile_pairs(const int32_t* cu, int64_t dq, int64_t qa, int64_t qb, int64_t ka, int64_t kb) {
  int64_t total = 0;
  for (int64_t d = dq;; ++d) {
    const int64_t s = cu[d], e = cu[d + 1];  // document d covers [s, e)
    if (e > s) {
      const int64_t ra = std::max(qa, s), rb = std::min(qb, e - 1);
      if (ra <= rb) {
        const int64_t lo = std::max(s, ka);  // first key any row of this segment may use
        // rows i <= kb contribute i - lo + 1 (when i >= lo)
        const int64_t a1 = std::max(ra, lo), b1 = std::min(rb, kb);
        if (a1 <= b1) total += ((a1 - lo + 1) + (b1 - lo + 1)) * (b1 - a1 + 1) / 2;
        // rows i > kb contribute kb - lo + 1 (when kb >= lo)
        const int64_t a2 = std::max(ra, kb + 1);
        if (a2 <= rb && kb >= lo) total += (rb - a2 + 1) * (kb - lo + 1);
      }
    }
    if (e - 1 >= qb) break;
  }
  return total;
}

// cu_seqlens: 0 = cu[0] <= ... <= cu[num_docs] = N
hsap_status check_cu(const int32_t* cu, int32_t num_docs, const Geom& g) {
  if (!cu) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (num_docs < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_docs %d < 1", num_docs);
  if (cu[0] != 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "cu_seqlens[0] = %d, expected 0", cu[0]);
  for (int32_t i = 0; i < num_docs; ++i)
    if (cu[i + 1] < cu[i]) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "cu_seqlens decreases at %d", i + 1);
  if ((int64_t)cu[num_docs] != g.N)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "cu_seqlens[%d] = %d, expected total_tokens x batch = %lld", num_docs,
              cu[num_docs], (long long)g.N);
  // documents stay inside their sequence: every sequence start is a document boundary
  for (int32_t b = 1; b < g.B; ++b)
    if (!std::binary_search(cu, cu + num_docs + 1, (int32_t)(b * g.Ns)))
      HSAP_FAIL(HSAP_ERR_INVALID_ARG, "sequence %d starts at %lld, which is not a document boundary", b,
                (long long)(b * g.Ns));
  return HSAP_OK;
}

// The non-empty tiles of one shard (validated geometry and cu_seqlens) in canonical order: stores
// the first `capacity` of them when `tiles` is not NULL and returns how many there are.
int64_t plan_shard(const int32_t* cu, int32_t num_docs, const Geom& g, const hsap_shard_desc& shard, hsap_tile* tiles,
                   int64_t capacity, int64_t* step_offsets, int64_t* useful_pairs) {
  const int32_t P = g.P, r = shard.shard_id;
  const int64_t BM = shard.block_m, BN = shard.block_n;
  const int64_t full = BM * BN;
  std::vector<Piece> qp, kp;
  shard_pieces(g, r, qp);
  const int pps = pieces_per_sequence(g);
  const bool store = tiles != nullptr;
  int64_t count = 0;
  if (step_offsets) step_offsets[0] = 0;
  for (int32_t step = 0; step < P; ++step) {
    const int32_t c = ((r - step) % P + P) % P;
    shard_pieces(g, c, kp);
    int64_t step_pairs = 0;
    for (int qi = 0; qi < (int)qp.size(); ++qi) {
      for (int64_t l0 = 0; l0 < qp[qi].len; l0 += BM) {
        const int64_t qa = qp[qi].global0 + l0, qb = qa + BM - 1;
        const int64_t q_tile = (qp[qi].local0 + l0) / BM;
        const int64_t dq = doc_of(cu, num_docs, qa);
        const int64_t s_first = cu[dq];
        const int64_t s_last = cu[doc_of(cu, num_docs, qb)];
        const int seq = qi / pps;  // keys of other sequences are never allowed
        for (int ki = seq * pps; ki < (seq + 1) * pps; ++ki) {
          const int64_t pa = kp[ki].global0, pb = pa + kp[ki].len - 1;
          const int64_t x = std::max(s_first, pa), y = std::min(qb, pb);
          if (x > y) continue;
          const int64_t u0 = (kp[ki].local0 + (x - pa)) / BN, u1 = (kp[ki].local0 + (y - pa)) / BN;
          for (int64_t u = u0; u <= u1; ++u) {
            const int64_t ka = pa + (u * BN - kp[ki].local0), kb = ka + BN - 1;
            const bool is_full = s_last <= ka && kb <= qa;
            const int64_t pairs = is_full ? full : tile_pairs(cu, dq, qa, qb, ka, kb);
            if (pairs == 0) continue;
            if (store && count < capacity)
              tiles[count] = hsap_tile{c, (int32_t)q_tile, (int32_t)u, pairs == full ? HSAP_TILE_FULL : HSAP_TILE_MASKED};
            ++count;
            step_pairs += pairs;
          }
        }
      }
    }
    if (step_offsets) step_offsets[step + 1] = count;
    if (useful_pairs) useful_pairs[step] = step_pairs;
  }
  return count;
}

}  // namespace
}  // namespace hsap

using namespace hsap;

extern "C" {

const char* hsap_status_string(hsap_status status) {
  switch (status) {
    case HSAP_OK: return "HSAP_OK";
    case HSAP_ERR_INVALID_ARG: return "HSAP_ERR_INVALID_ARG";
    case HSAP_ERR_CAPACITY: return "HSAP_ERR_CAPACITY";
    case HSAP_ERR_UNSUPPORTED: return "HSAP_ERR_UNSUPPORTED";
    case HSAP_ERR_HIP: return "HSAP_ERR_HIP";
  }
  return "HSAP_ERR_UNKNOWN";
}

const char* hsap_last_error(void) { return g_last_error.c_str(); }

hsap_status hsap_plan(const int32_t* cu, int32_t num_docs, const hsap_shard_desc* shard, hsap_tile* tiles,
                      int64_t capacity, int64_t* num_tiles, int64_t* step_offsets, int64_t* useful_pairs) {
  clear_error();
  Geom g;
  hsap_status st = check_shard(shard, &g);
  if (st != HSAP_OK) return st;
  if (!num_tiles) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_tiles is NULL");
  if (capacity < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "capacity < 0");
  st = check_cu(cu, num_docs, g);
  if (st != HSAP_OK) return st;
  const int64_t count = plan_shard(cu, num_docs, g, *shard, tiles, capacity, step_offsets, useful_pairs);
  *num_tiles = count;
  if (!tiles || count > capacity)
    HSAP_FAIL(HSAP_ERR_CAPACITY, "tile list needs %lld entries, capacity %lld", (long long)count, (long long)capacity);
  return HSAP_OK;
}

hsap_status hsap_load_matrix(const int32_t* cu, int32_t num_docs, const hsap_shard_desc* shard, int64_t* tiles,
                             int64_t* pairs) {
  clear_error();
  if (!shard) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "shard descriptor is NULL");
  if (!tiles && !pairs) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "tiles and pairs are both NULL");
  hsap_shard_desc sd = *shard;
  sd.shard_id = 0;  // every shard is planned; only the geometry of the descriptor is used
  Geom g;
  hsap_status st = check_shard(&sd, &g);
  if (st != HSAP_OK) return st;
  st = check_cu(cu, num_docs, g);
  if (st != HSAP_OK) return st;
  const int32_t P = g.P;
  std::vector<int64_t> offs((size_t)P + 1), step_pairs((size_t)P);
  for (int32_t r = 0; r < P; ++r) {
    sd.shard_id = r;
    plan_shard(cu, num_docs, g, sd, nullptr, 0, offs.data(), step_pairs.data());
    for (int32_t step = 0; step < P; ++step) {
      const int32_t c = ((r - step) % P + P) % P;
      if (tiles) tiles[(int64_t)r * P + c] = offs[(size_t)step + 1] - offs[(size_t)step];
      if (pairs) pairs[(int64_t)r * P + c] = step_pairs[(size_t)step];
    }
  }
  return HSAP_OK;
}

hsap_status hsap_balance(int32_t sp_degree, const int64_t* cost, int32_t* exec_rank, int64_t* load) {
  clear_error();
  if (sp_degree < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "sp_degree %d < 1", sp_degree);
  if (!cost || !exec_rank) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL cost or exec_rank");
  const int64_t P = sp_degree;
  for (int64_t i = 0; i < P * P; ++i)
    if (cost[i] < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "cost[%lld] < 0", (long long)i);
  // ring assignment: every block on its shard's rank
  std::vector<int64_t> ld((size_t)P, 0);
  for (int32_t r = 0; r < P; ++r)
    for (int32_t c = 0; c < P; ++c) {
      exec_rank[r * P + c] = r;
      ld[(size_t)r] += cost[r * P + c];
    }
  // The most loaded rank (lowest index among equals) hands one block to the block's other
  // eligible rank while the receiver stays below the giver's load; the move leaving the smaller
  // maximum of the two loads wins (equal: lower r, then lower c).  Each move lowers the sum of
  // squared loads, so the loop ends.
  for (;;) {
    int32_t g = 0;
    for (int32_t e = 1; e < P; ++e)
      if (ld[(size_t)e] > ld[(size_t)g]) g = e;
    int64_t best_key = -1;
    int32_t best_r = -1, best_c = -1, best_t = -1;
    auto consider = [&](int32_t r, int32_t c) {
      const int64_t w = cost[r * P + c];
      if (r == c || w == 0 || exec_rank[r * P + c] != g) return;
      const int32_t t = g == r ? c : r;
      if (ld[(size_t)t] + w >= ld[(size_t)g]) return;
      const int64_t key = std::max(ld[(size_t)g] - w, ld[(size_t)t] + w);
      // (key, r, c) lexicographic; candidates arrive in increasing (r, c) order below
      if (best_key < 0 || key < best_key) {
        best_key = key;
        best_r = r;
        best_c = c;
        best_t = t;
      }
    };
    // blocks rank g may hold: its own row (g, c) and transferred blocks (r, g), in (r, c) order
    for (int32_t r = 0; r < P; ++r) {
      if (r == g)
        for (int32_t c = 0; c < P; ++c) consider(g, c);
      else
        consider(r, g);
    }
    if (best_key < 0) break;
    const int64_t w = cost[best_r * P + best_c];
    exec_rank[best_r * P + best_c] = best_t;
    ld[(size_t)g] -= w;
    ld[(size_t)best_t] += w;
  }
  if (load) std::copy(ld.begin(), ld.end(), load);
  return HSAP_OK;
}

hsap_status hsap_plan_runs(const hsap_shard_desc* shard, const hsap_tile* tiles, int64_t num_tiles, int32_t major,
                           int32_t max_run_tiles, hsap_tile* sorted_tiles, hsap_run* runs, int64_t capacity,
                           int64_t* num_runs, int32_t* num_slots) {
  clear_error();
  Geom g;
  hsap_status st = check_shard(shard, &g);
  if (st != HSAP_OK) return st;
  if (major != HSAP_MAJOR_Q && major != HSAP_MAJOR_K && major != HSAP_MAJOR_Q_ALL)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "unknown major %d", major);
  if (num_tiles < 0 || (num_tiles > 0 && !tiles)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "tiles is NULL");
  if (num_tiles > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many tiles");
  if (!num_runs) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_runs is NULL");
  if (num_tiles > 0 && !sorted_tiles) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "sorted_tiles is NULL");
  if (capacity < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "capacity < 0");
  const int32_t P = g.P, r = shard->shard_id;
  const int64_t nq = g.n / shard->block_m, nk = g.n / shard->block_n;
  std::vector<int32_t> step_tab(P);  // ring step at which shard r holds chunk c
  for (int32_t c = 0; c < P; ++c) step_tab[c] = ((r - c) % P + P) % P;
  auto step_of = [&](int32_t c) { return step_tab[c]; };
  // the list must be canonical: ring step, q_tile, k_tile strictly increasing
  for (int64_t i = 0; i < num_tiles; ++i) {
    const hsap_tile& t = tiles[i];
    if (t.chunk < 0 || t.chunk >= P || t.q_tile < 0 || t.q_tile >= nq || t.k_tile < 0 || t.k_tile >= nk ||
        (t.kind != HSAP_TILE_FULL && t.kind != HSAP_TILE_MASKED))
      HSAP_FAIL(HSAP_ERR_INVALID_ARG, "tile %lld out of range", (long long)i);
    if (i > 0) {
      const hsap_tile& p = tiles[i - 1];
      const int64_t a = ((int64_t)step_of(p.chunk) * nq + p.q_tile) * nk + p.k_tile;
      const int64_t b = ((int64_t)step_of(t.chunk) * nq + t.q_tile) * nk + t.k_tile;
      if (b <= a) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "tile list not in canonical order at %lld", (long long)i);
    }
  }
  // Stable counting sort of tiles[lo, hi) by `bucket` into sorted_tiles[lo, hi).  The
  // canonical list is ordered by (ring step, q_tile, k_tile), so a stable pass by q_tile
  // over the whole list orders by (q_tile, ring step, k_tile), and one by k_tile within
  // each ring step's segment orders that segment by (k_tile, q_tile).
  std::vector<int64_t> bucket_at;
  auto counting_sort = [&](int64_t lo, int64_t hi, int64_t buckets, auto bucket) {
    bucket_at.assign((size_t)buckets + 1, 0);
    for (int64_t i = lo; i < hi; ++i) ++bucket_at[(size_t)bucket(tiles[i]) + 1];
    for (int64_t b = 0; b < buckets; ++b) bucket_at[(size_t)b + 1] += bucket_at[(size_t)b];
    for (int64_t i = lo; i < hi; ++i) sorted_tiles[lo + bucket_at[(size_t)bucket(tiles[i])]++] = tiles[i];
  };
  std::vector<hsap_run> out;
  int32_t slots = 0;
  if (major == HSAP_MAJOR_Q) {
    if (num_tiles > 0) std::memcpy(sorted_tiles, tiles, sizeof(hsap_tile) * num_tiles);
    const int64_t max_run = max_run_tiles > 0 ? max_run_tiles : INT64_MAX;
    auto pieces_for = [&](int64_t cnt) { return cnt == 0 ? 0 : (cnt - 1) / max_run + 1; };  // no overflow
    int64_t i = 0;
    std::vector<int64_t> first(nq), count(nq);
    while (i < num_tiles) {
      const int32_t c = tiles[i].chunk;
      // per q-tile extent of this chunk's tiles, and the pieces the longest needs
      int64_t pieces = 1;
      for (int32_t t = 0; t < nq; ++t) {
        int64_t j = i;
        while (j < num_tiles && tiles[j].chunk == c && tiles[j].q_tile == t) ++j;
        first[t] = i;
        count[t] = j - i;
        pieces = std::max<int64_t>(pieces, pieces_for(count[t]));
        i = j;
      }
      // every q-tile gets a run in every slot the chunk uses (count 0 where it has nothing there)
      for (int32_t t = 0; t < nq; ++t) {
        const int64_t need = std::max<int64_t>(1, pieces_for(count[t]));
        int64_t at = first[t];
        for (int64_t piece = 0; piece < pieces; ++piece) {
          int64_t len = 0;
          if (piece < need) len = count[t] / need + (piece < count[t] % need ? 1 : 0);
          out.push_back(hsap_run{(int32_t)(c + P * piece), t, (int32_t)at, (int32_t)len});
          at += len;
        }
      }
      slots = std::max<int32_t>(slots, (int32_t)(c + P * (pieces - 1) + 1));
    }
  } else if (major == HSAP_MAJOR_Q_ALL) {
    counting_sort(0, num_tiles, nq, [](const hsap_tile& t) { return t.q_tile; });
    int64_t i = 0;
    for (int32_t t = 0; t < nq; ++t) {
      int64_t j = i;
      while (j < num_tiles && sorted_tiles[j].q_tile == t) ++j;
      out.push_back(hsap_run{0, t, (int32_t)i, (int32_t)(j - i)});
      i = j;
    }
    slots = 1;
  } else {
    for (int64_t lo = 0; lo < num_tiles;) {  // one ring step (one chunk) at a time
      int64_t hi = lo;
      while (hi < num_tiles && tiles[hi].chunk == tiles[lo].chunk) ++hi;
      counting_sort(lo, hi, nk, [](const hsap_tile& t) { return t.k_tile; });
      lo = hi;
    }
    int64_t i = 0;
    while (i < num_tiles) {
      int64_t j = i;
      while (j < num_tiles && sorted_tiles[j].chunk == sorted_tiles[i].chunk &&
             sorted_tiles[j].k_tile == sorted_tiles[i].k_tile)
        ++j;
      out.push_back(hsap_run{sorted_tiles[i].chunk, sorted_tiles[i].k_tile, (int32_t)i, (int32_t)(j - i)});
      slots = std::max<int32_t>(slots, sorted_tiles[i].chunk + 1);
      i = j;
    }
  }
  // longest first; ties by ring step, tile, then slot, so the order is unique
  std::stable_sort(out.begin(), out.end(), [&](const hsap_run& a, const hsap_run& b) {
    if (a.count != b.count) return a.count > b.count;
    const int32_t sa = step_of(a.slot % P), sb = step_of(b.slot % P);
    if (sa != sb) return sa < sb;
    if (a.tile != b.tile) return a.tile < b.tile;
    return a.slot < b.slot;
  });
  *num_runs = (int64_t)out.size();
  if (num_slots) *num_slots = slots;
  if (!runs || (int64_t)out.size() > capacity)
    HSAP_FAIL(HSAP_ERR_CAPACITY, "run list needs %lld entries, capacity %lld", (long long)out.size(),
              (long long)capacity);
  std::copy(out.begin(), out.end(), runs);
  return HSAP_OK;
}

int32_t hsap_split_length(const hsap_shard_desc* shard, int64_t num_tiles, int32_t heads_q,
                          int32_t resident_workgroups) {
  clear_error();
  Geom g;
  if (check_shard(shard, &g) != HSAP_OK) return -1;
  if (num_tiles < 0 || heads_q <= 0 || resident_workgroups <= 0) {
    set_error("bad num_tiles, heads_q or resident_workgroups");
    return -1;
  }
  const int64_t nk = g.ns / shard->block_n;  // a run never leaves its sequence
  const int64_t avg = (num_tiles * heads_q + resident_workgroups - 1) / resident_workgroups;
  if (nk <= avg) return 0;  // no run can exceed the average load
  const int64_t len = std::max<int64_t>({avg, 4, (nk + 3) / 4});
  return len >= nk ? 0 : (int32_t)len;
}

}  // extern "C"
