// Partial attention backward: gradients of one shard's attention with
// respect to its queries and to the listed k-tiles of each K/V chunk (the
// backward "computing" whose results the paper's per-rank code returns as dq
// and dkv messages, instruction table of the SAP section).  P is recomputed
// from the final (merged) LSE, so no attention matrix is stored between
// forward and backward.  Two kernels share the work, so that neither needs
// atomics per k-tile:
//
// dK/dV kernels: one workgroup per (k-major run, K/V head).  A run is one
// (chunk, k-tile) with the q-tiles listed against it; the workgroup keeps the
// k-tile's K and V rows (as MFMA B operands) and its dK, dV accumulators in
// registers for the whole run, looping over the query heads of its K/V head
// group and over the listed q-tiles in sub-tiles of 64 rows.  Per sub-tile:
//   S  = Q K^T, dP = dO V^T           (lane = key, registers = queries)
//   P  = exp2(S * scale*log2e - LSE*log2e) on allowed pairs, dS = P (dP - delta)
//   dV += P^T dO, dK += dS^T Q        (A operands from registers; dO and Q
//                                      read transposed from LDS)
// For head_dim 128 with 128-key tiles (every benchmark workload) the split
// kernel gives each 32-key block to two waves on one SIMD, one forming S, P
// and dV, the other dP, dS and dK (P handed over through LDS); otherwise one
// wave owns 32 keys and does all four products.  Q and dO sub-tiles sit in
// XOR-swizzled LDS tiles (mfma.h).  Each (chunk, k-tile, K/V head) block of
// dK/dV has one owner.
//
// dQ kernel: one workgroup per (q-major run, query head), shaped like the
// forward; it forms S and dP again for its own pairs (described below).
//
#include <type_traits>

#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

struct BwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* d_o;
  const float* lse;
  const float* delta;
  const __bf16* o;     // when set, the dQ kernel computes delta from O and dO itself, writing delta_out
  float* delta_out;
  const int32_t* doc_start;
  const hsap_tile* tiles;
  const hsap_run* runs;
  float* dq;       // fp32 accumulators (+=), or
  float* dk;
  float* dv;
  __bf16* dq16;    // final bf16 gradients (written once)
  __bf16* dk16;
  __bf16* dv16;
  Geom geom;
  int32_t shard;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t bm;
  float scale;
  float scale_log2;
  int32_t num_tiles;     // tile-list mode: entries of tiles (one chunk's, sorted by q_tile)
  int32_t chunk;         // tile-list mode: the chunk of every tile
};

// Tile-list mode of the dK/dV kernel: at most this many q-tiles (n / BM) per k-tile.
constexpr int kMaxListQTiles = 2048;

template <int D, int WAVES, bool BF16OUT, bool LIST = false>
__global__ __launch_bounds__(64 * WAVES, 1) void attn_bwd_dkdv_kernel(BwdArgs a) {
  static_assert(!LIST || !BF16OUT, "the tile-list mode accumulates fp32");
  constexpr int BN = 32 * WAVES;
  constexpr int NT = 64 * WAVES;
  constexpr int SUB = 64;                 // query rows per sub-tile
  constexpr int CPR = D / 8;              // 16-byte chunks per Q / dO / K row
  constexpr int MB = D / 32;              // 32-wide blocks of d
  constexpr int PER_T = SUB * CPR / NT;   // chunks of Q (and of dO) per thread per sub-tile
  static_assert((SUB * CPR) % NT == 0 && (BN * CPR) % NT == 0, "tiles must split evenly over the threads");
  static_assert(D == 128 || D == 64, "head_dim 64 or 128");
  constexpr float LOG2E = 1.44269504088896340736f;
  __shared__ __attribute__((aligned(16))) __bf16 Qs[2][SUB * D];
  __shared__ __attribute__((aligned(16))) __bf16 dOs[2][SUB * D];
  __shared__ __attribute__((aligned(16))) float lse_s[2][SUB];
  __shared__ __attribute__((aligned(16))) float delta_s[2][SUB];
  __shared__ __attribute__((aligned(16))) int32_t start_s[2][SUB];
  __shared__ uint32_t qlist[LIST ? kMaxListQTiles : 1];  // tile-list mode: this k-tile's q-tiles (q_tile | kind << 31)
  __shared__ int32_t wave_hits[WAVES];

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int run_idx = blockIdx.x / a.hkv;
  const int g = blockIdx.x - run_idx * a.hkv;
  // Run mode: a k-major run from hsap_plan_runs (never empty).  Tile-list mode: k-tile run_idx of
  // chunk a.chunk; the workgroup gathers the tiles with that k_tile from the list (sorted by
  // q_tile) into LDS, in list order, 64 per wave per pass.
  constexpr bool list_mode = LIST;
  const hsap_run run = list_mode ? hsap_run{a.chunk, run_idx, 0, 0} : a.runs[run_idx];
  const int c = list_mode ? a.chunk : a.tiles[run.first].chunk;
  int count = run.count;
  if (list_mode) {
    int total = 0;
    for (int base = 0; base < a.num_tiles; base += 64 * WAVES) {
      const int i = base + 64 * w + lane;
      bool hit = false;
      uint32_t packed = 0u;
      if (i < a.num_tiles) {
        const hsap_tile t = a.tiles[i];
        hit = t.k_tile == run.tile;
        packed = (uint32_t)t.q_tile | ((uint32_t)t.kind << 31);
      }
      const uint64_t m = __builtin_amdgcn_ballot_w64(hit);
      const int rank = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (lane == 0) wave_hits[w] = __popcll(m);
      __syncthreads();
      int off = total, all = 0;
      for (int x = 0; x < WAVES; ++x) {
        off += x < w ? wave_hits[x] : 0;
        all += wave_hits[x];
      }
      if (hit && off + rank < kMaxListQTiles) qlist[off + rank] = packed;
      total += all;
      __syncthreads();  // wave_hits is rewritten by the next pass; qlist is complete after the last
    }
    count = min(total, kMaxListQTiles);
    if (count == 0) return;  // no query of the shard reaches this k-tile in the chunk: nothing to add
  }
  const int64_t n = a.geom.n;
  const int64_t krow0 = (int64_t)run.tile * BN;
  const int32_t gk = (int32_t)global_pos(a.geom, c, krow0 + 32 * w + l32);  // this lane's key position
  const int64_t kvrow = (int64_t)c * n + krow0;                            // first row in the sharded K/V buffers

  // ---- LDS offsets (elements) as lane constants + compile-time immediates -------------
  // Row reads (row 32 qb + l32, chunk 2 kk + hi) of a swizzled [rows][D] tile:
  //   offset = 32 qb * D + rowoff[kk]
  // Transpose reads (rows rb + tr_row with rb = 8 k (mod 16), columns 32 mb + tr_col):
  //   offset = rb * D + troff[mb][k]      (the swizzle of rb + tr_row depends on k only)
  const int tr_row = 4 * hi + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int rowoff[D / 16], troff[MB][2];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) rowoff[kk] = swz<CPR>(l32, 16 * kk + 8 * hi);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int k = 0; k < 2; ++k) troff[mb][k] = swz<CPR>(8 * k + tr_row, 32 * mb + tr_col) - 8 * k * D;

  // K and V rows of this lane's key as MFMA B operands
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const int64_t off = ((kvrow + 32 * w + l32) * a.hkv + g) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      kf[kk] = *(const bf16x8*)(a.k + off + 16 * kk);
      vf[kk] = *(const bf16x8*)(a.v + off + 16 * kk);
    }
  }

  f32x16 dk[MB], dv[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    dk[mb] = f32x16{};
    dv[mb] = f32x16{};
  }

  const int nsub = a.bm / SUB;
  const int per_head = count * nsub;
  const int total = a.group * per_head;
  // The run's q-tiles, packed one per lane (q_tile | kind << 31) in windows of 64 tiles, read
  // with v_readlane: the next sub-tile's address never waits on a memory load.  Window v lives
  // in win0 (v even) or win1 (v odd); sub-tiles visit the run's tiles in order once per query
  // head, so the window is reloaded when the tile index leaves it.
  uint32_t win0 = 0u, win1 = 0u;
  int win_lo = 0, win_hi = -1;  // windows held: win_lo (and win_lo + 1 when win_hi > win_lo)
  auto load_window = [&](int v) {
    const int i = 64 * v + lane;
    uint32_t p = 0;
    if (i < count) {
      if (!list_mode) {
        const hsap_tile t = a.tiles[run.first + i];
        p = (uint32_t)t.q_tile | ((uint32_t)t.kind << 31);
      } else {
        p = qlist[i];
      }
    }
    if (v & 1) win1 = p;
    else win0 = p;
  };
  auto ensure_window = [&](int v) {  // v is the window of the next tile index needed
    if (v >= win_lo && v <= win_hi) return;
    load_window(v);
    if (v == win_hi + 1 && v - 1 >= win_lo) win_lo = v - 1;
    else win_lo = v;
    win_hi = v;
  };
  // sub-tile `it`: query head, tile of the run (packed), 64-row slice of the tile
  auto head_of = [&](int it) { return g * a.group + it / per_head; };
  auto tile_of = [&](int it) -> uint32_t {
    const int idx = (it % per_head) / nsub;
    return __builtin_amdgcn_readlane(((idx >> 6) & 1) ? win1 : win0, idx & 63);
  };
  auto q0_of = [&](uint32_t t, int it) {
    return (int64_t)(t & 0x7FFFFFFFu) * a.bm + ((it % per_head) % nsub) * SUB;
  };
  ensure_window(0);

  // staging of one sub-tile: Q and dO rows, and the per-row LSE, delta and document start
  int32_t soff[PER_T], loff[PER_T];
#pragma unroll
  for (int i = 0; i < PER_T; ++i) {
    const int idx = tid + i * NT, row = idx / CPR, cc = idx % CPR;
    soff[i] = row * a.hq * D + cc * 8;
    loff[i] = swz<CPR>(row, cc * 8);
  }
  bf16x8 qreg[PER_T], oreg[PER_T];
  float lreg = 0.f, dreg = 0.f;
  int32_t sreg = 0;
  auto load_sub = [&](int it) {
    const int h = head_of(it);
    ensure_window(((it % per_head) / nsub) >> 6);
    const uint32_t t = tile_of(it);
    const int64_t q0 = q0_of(t, it);
    const int64_t base = (q0 * a.hq + h) * D;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      qreg[i] = *(const bf16x8*)(a.q + base + soff[i]);
      oreg[i] = *(const bf16x8*)(a.d_o + base + soff[i]);
    }
    if (tid < SUB) {
      lreg = a.lse[(int64_t)h * n + q0 + tid];
      dreg = a.delta[(int64_t)h * n + q0 + tid];
      sreg = a.doc_start[global_pos(a.geom, a.shard, q0) + tid];
    }
  };
  auto store_sub = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      *(bf16x8*)(&Qs[buf][loff[i]]) = qreg[i];
      *(bf16x8*)(&dOs[buf][loff[i]]) = oreg[i];
    }
    if (tid < SUB) {
      lse_s[buf][tid] = lreg == -__builtin_inff() ? __builtin_inff() : lreg * LOG2E;  // no key: P = 0
      delta_s[buf][tid] = dreg;
      start_s[buf][tid] = sreg;
    }
  };

  load_sub(0);
  store_sub(0);
  __syncthreads();

  for (int it = 0; it < total; ++it) {
    const int buf = it & 1;
    const int h = head_of(it);
    const uint32_t tile = tile_of(it);
    const int64_t q0 = q0_of(tile, it);
    const int32_t gq0 = (int32_t)global_pos(a.geom, a.shard, q0);
    const bool masked = (tile >> 31) != 0;
    if (it + 1 < total) load_sub(it + 1);
    const __bf16* Q = Qs[buf];
    const __bf16* O = dOs[buf];

    // per block of 32 queries: S = Q K^T, dP = dO V^T (register j = query 32 qb + c_row(j, hi)),
    // then P and dS, then dV += P^T dO and dK += dS^T Q, then dS^T to LDS
#pragma unroll
    for (int qb = 0; qb < SUB / 32; ++qb) {
      f32x16 sacc{}, dpacc{};
      bf16x8 qa[D / 16], oa[D / 16];  // all operand reads of the block first, then the MFMAs
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        qa[kk] = *(const bf16x8*)(Q + 32 * qb * D + rowoff[kk]);
        oa[kk] = *(const bf16x8*)(O + 32 * qb * D + rowoff[kk]);
      }
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        sacc = mfma32(qa[kk], kf[kk], sacc);
        dpacc = mfma32(oa[kk], vf[kk], dpacc);
      }
      // the transposed dO and Q reads of the dV / dK products depend on no score: issued here, they
      // land while P and dS are computed (one wave per SIMD has nothing else to hide them)
      bf16x8 bo[2][MB], bq[2][MB];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int rb = (32 * qb + 16 * half) * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          bo[half][mb] = cat4(ds_read_tr16(O + rb + troff[mb][0]), ds_read_tr16(O + rb + 8 * D + troff[mb][1]));
          bq[half][mb] = cat4(ds_read_tr16(Q + rb + troff[mb][0]), ds_read_tr16(Q + rb + 8 * D + troff[mb][1]));
        }
      }
      // P for the block (register j = 4 grp + e holds query q4 + e, q4 = 32 qb + 8 grp + 4 hi),
      // masked in one uniform branch, then P and dS = P (dP - delta) as bf16
      float p[16];
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const f32x4 l4 = *(const f32x4*)(&lse_s[buf][32 * qb + 8 * grp + 4 * hi]);
#pragma unroll
        for (int e = 0; e < 4; ++e) p[4 * grp + e] = fast_exp2(__builtin_fmaf(sacc[4 * grp + e], a.scale_log2, -l4[e]));
      }
      if (masked) {
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const int q4 = 32 * qb + 8 * grp + 4 * hi;
          const i32x4 s4 = *(const i32x4*)(&start_s[buf][q4]);
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if ((uint32_t)(gk - s4[e]) > (uint32_t)(gq0 + q4 + e - s4[e])) p[4 * grp + e] = 0.f;
        }
      }
      bf16x8 pb[2], sb[2];
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const f32x4 d4 = *(const f32x4*)(&delta_s[buf][32 * qb + 8 * grp + 4 * hi]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = 4 * grp + e;
          pb[j >> 3][j & 7] = (__bf16)p[j];
          sb[j >> 3][j & 7] = (__bf16)(p[j] * (dpacc[j] - d4[e]));
        }
      }
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          dv[mb] = mfma32(pb[half], bo[half][mb], dv[mb]);
          dk[mb] = mfma32(sb[half], bq[half][mb], dk[mb]);
        }
    }

    if (it + 1 < total) store_sub(buf ^ 1);
    hsap_lds_barrier();
  }

  // this workgroup owns rows [krow0, krow0 + BN) of chunk c for K/V head g: plain read-add-write
  // of the fp32 accumulators, or a store of the final bf16 values
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t idx = ((kvrow + 32 * w + c_row(j, hi)) * a.hkv + g) * D + 32 * mb + l32;
      if (BF16OUT) {
        a.dk16[idx] = (__bf16)(dk[mb][j] * a.scale);
        a.dv16[idx] = (__bf16)dv[mb][j];
      } else {
        a.dk[idx] += dk[mb][j] * a.scale;
        a.dv[idx] += dv[mb][j];
      }
    }
}

// ---------------------------------------------------------------------------
// dK/dV kernel with split roles (head_dim 128, BN = 128): eight waves, two per
// key block of 32 keys.  Wave kb (0..3) is the block's S wave: it holds the
// block's K rows as MFMA B operands and its dV accumulators; wave 4 + kb is
// the dP wave: V rows and dK accumulators.  Per 64-row q sub-tile:
//   scores    S wave:  S = Q K^T, P = exp2(S * scale*log2e - LSE*log2e) on
//                      allowed pairs; P (fp16) to LDS for its partner
//             dP wave: dP = dO V^T
//   products  S wave:  dV += P^T dO             (dO read transposed)
//             dP wave: P from LDS, dS = P (dP - delta), dK += dS^T Q
//                      (Q read transposed)
// software-pipelined by one sub-tile: iteration t runs the products of t and
// the scores of t + 1, with one barrier, while the Q and dO rows of t + 2 go
// from global memory straight into LDS (global_load_lds).
// Each wave issues 32 MFMAs per sub-tile, half of the one-wave-per-block
// kernel's 64, and holds half its state (K or V, dK or dV), so two waves fit
// on a SIMD: one wave's exponentials (or dS arithmetic) run while the other
// wave's products occupy the matrix core.  S and dP are formed once.
// Wave w and wave w + 4 share a SIMD (waves are placed round-robin).
// ---------------------------------------------------------------------------
template <bool BF16OUT>
__global__ __launch_bounds__(512, 2) void attn_bwd_dkdv_split_kernel(BwdArgs a) {
  constexpr int D = 128, WAVES = 8, KB = 4;  // KB key blocks of 32: BN = 128
  constexpr int NT = 64 * WAVES;
  constexpr int SUB = 64;
  constexpr int CPR = D / 8;
  constexpr int MB = D / 32;
  constexpr int WCH = SUB * CPR / WAVES;       // 16-byte chunks of a Q (or dO) sub-tile a wave moves
  constexpr int U = WCH / 64;                   // transfer instructions per wave per sub-tile and tensor
  static_assert(WCH % 64 == 0, "a wave moves whole instructions of a sub-tile");
  constexpr float LOG2E = 1.44269504088896340736f;
  // a ring of three sub-tiles: t (gradient products), t + 1 (scores), t + 2 (in flight)
  __shared__ __attribute__((aligned(16))) __bf16 Qs[3][SUB * D];
  __shared__ __attribute__((aligned(16))) __bf16 dOs[3][SUB * D];
  __shared__ __attribute__((aligned(16))) float lse_s[3][SUB];
  __shared__ __attribute__((aligned(16))) float ndelta_s[3][SUB];  // -delta
  __shared__ __attribute__((aligned(16))) int32_t start_s[3][SUB];
  // P hand-off in fp16 (two buffers: P of sub-tile t + 1 is written while the dP wave reads P of
  // t), per key block and 32-query block: lane l's 16 values as two 16-byte pieces at [half][l]
  // (consecutive lanes at consecutive 16 bytes: no bank conflict)
  __shared__ __attribute__((aligned(16))) h16x8 Px[2][KB][SUB / 32][2][64];
  typedef __attribute__((address_space(3))) void* lds_void;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const bool s_wave = w < KB;               // wave-uniform role
  const int kb = s_wave ? w : w - KB;       // key block
  const int run_idx = blockIdx.x / a.hkv;
  const int g = blockIdx.x - run_idx * a.hkv;
  const hsap_run run = a.runs[run_idx];
  const int c = a.tiles[run.first].chunk;  // k-major runs are never empty
  const int count = run.count;
  const int64_t n = a.geom.n;
  const int64_t krow0 = (int64_t)run.tile * (32 * KB);
  const int32_t gk = (int32_t)global_pos(a.geom, c, krow0 + 32 * kb + l32);  // this lane's key position
  const int64_t kvrow = (int64_t)c * n + krow0;

  // row reads (row 32 qb + l32, chunk 2 kk + hi) and transpose reads of the swizzled tiles, as in
  // the one-wave-per-block kernel
  const int tr_row = 4 * hi + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int rowoff[D / 16], troff[MB][2];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) rowoff[kk] = swz<CPR>(l32, 16 * kk + 8 * hi);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int k = 0; k < 2; ++k) troff[mb][k] = swz<CPR>(8 * k + tr_row, 32 * mb + tr_col) - 8 * k * D;

  // this lane's key row of K (S wave) or V (dP wave) as MFMA B operands
  bf16x8 kv[D / 16];
  {
    const __bf16* src = s_wave ? a.k : a.v;
    const int64_t off = ((kvrow + 32 * kb + l32) * a.hkv + g) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) kv[kk] = *(const bf16x8*)(src + off + 16 * kk);
  }
  f32x16 acc[MB];  // dV (S wave) or dK (dP wave)
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x16{};

  const int nsub = a.bm / SUB;
  const int total = a.group * count * nsub;
  uint32_t win0 = 0u, win1 = 0u;
  int win_lo = 0, win_hi = -1;
  auto load_window = [&](int v) {
    const int i = 64 * v + lane;
    uint32_t p = 0;
    if (i < count) {
      const hsap_tile t = a.tiles[run.first + i];
      p = (uint32_t)t.q_tile | ((uint32_t)t.kind << 31);
    }
    if (v & 1) win1 = p;
    else win0 = p;
  };
  auto ensure_window = [&](int v) {
    if (v >= win_lo && v <= win_hi) return;
    load_window(v);
    if (v == win_hi + 1 && v - 1 >= win_lo) win_lo = v - 1;
    else win_lo = v;
    win_hi = v;
  };
  // Sub-tile position as counters (no division in the loop): query head h, tile index idx in the
  // run, 64-row slice sb of the tile; the next sub-tile's counters advance one step at a time.
  struct Pos {
    int h, idx, sb;
  };
  auto advance = [&](Pos p) {
    if (++p.sb == nsub) {
      p.sb = 0;
      if (++p.idx == count) {
        p.idx = 0;
        ++p.h;
      }
    }
    return p;
  };
  auto tile_at = [&](const Pos& p) -> uint32_t {
    return __builtin_amdgcn_readlane(((p.idx >> 6) & 1) ? win1 : win0, p.idx & 63);
  };
  auto q0_at = [&](uint32_t t, const Pos& p) { return (int64_t)(t & 0x7FFFFFFFu) * a.bm + p.sb * SUB; };
  ensure_window(0);

  // Q and dO sub-tiles by direct-to-LDS transfers: instruction u of wave w fills chunk positions
  // p = WCH w + 64 u + lane of the swizzled tile; the lane's source is the chunk the swizzle places
  // there, a 32-bit byte offset from the sub-tile's scalar base (Q and dO rows have the same stride)
  uint32_t gsrc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int p = WCH * w + 64 * u + lane, row = p / CPR;
    gsrc[u] = (uint32_t)((row * a.hq * D + swz_chunk<CPR>(row, p % CPR) * 8) * 2);
  }
  const int wu = __builtin_amdgcn_readfirstlane(w);
  auto stage = [&](const __bf16* src, __bf16* dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_void)dst + (uint32_t)(WCH * wu * 16);
#pragma unroll
    for (int u = 0; u < U; ++u)
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(gsrc[u]), "s"(src), "{m0}"(lds + 64 * 16 * u));
  };
  float lreg = 0.f, dreg = 0.f;
  int32_t sreg = 0;
  // the sub-tile's Q and dO into buffer buf (transfers), its LSE, delta and document starts into
  // registers of the first 64 threads (written to LDS by store_sub)
  auto load_sub = [&](const Pos& ps, int buf) {
    const int h = g * a.group + ps.h;
    ensure_window(ps.idx >> 6);
    const uint32_t t = tile_at(ps);
    const int64_t q0 = q0_at(t, ps);
    const int64_t base = (q0 * a.hq + h) * D;
    stage(a.q + base, Qs[buf]);
    stage(a.d_o + base, dOs[buf]);
    if (tid < SUB) {
      lreg = a.lse[(int64_t)h * n + q0 + tid];
      dreg = a.delta[(int64_t)h * n + q0 + tid];
      sreg = a.doc_start[global_pos(a.geom, a.shard, q0) + tid];
    }
  };
  auto store_sub = [&](int buf) {
    if (tid < SUB) {
      lse_s[buf][tid] = lreg == -__builtin_inff() ? __builtin_inff() : lreg * LOG2E;  // no key: P = 0
      ndelta_s[buf][tid] = -dreg;
      start_s[buf][tid] = sreg;
    }
  };

  // Scores of a sub-tile from its rows (buffer rb): S = Q K^T (S wave) or dP = dO V^T (dP wave)
  // into sp; the S wave turns them into P (register j = 4 grp + e holds query q4 + e,
  // q4 = 32 qb + 8 grp + 4 hi; P = exp2(S * scale*log2e - LSE*log2e), masked in one uniform
  // branch), kept in bf16 as its own next A operand and handed to the dP wave in fp16.
  f32x16 sp[SUB / 32];
  bf16x8 opnd[SUB / 32][2];  // A operands of the gradient products: P (S wave) or dS (dP wave)
  auto scores = [&](int rb, int pbuf, bool masked, int32_t gq0) {
    const __bf16* R = s_wave ? Qs[rb] : dOs[rb];
#pragma unroll
    for (int qb = 0; qb < SUB / 32; ++qb) {
      bf16x8 ra[D / 16];
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) ra[kk] = *(const bf16x8*)(R + 32 * qb * D + rowoff[kk]);
      if (s_wave) {
        sp[qb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) sp[qb] = mfma32(ra[kk], kv[kk], sp[qb]);
      } else {
        // the products accumulate onto -delta of each query (register j = 4 cq + e), so the
        // chain ends with dP - delta and dS takes one multiply per element
        f32x16 init;
#pragma unroll
        for (int cq = 0; cq < 4; ++cq) {
          const f32x4 d4 = *(const f32x4*)(&ndelta_s[rb][32 * qb + 8 * cq + 4 * hi]);
#pragma unroll
          for (int e = 0; e < 4; ++e) init[4 * cq + e] = d4[e];
        }
        sp[qb] = init;
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) sp[qb] = mfma32(ra[kk], kv[kk], sp[qb]);
      }
    }
    if (s_wave) {
#pragma unroll
      for (int qb = 0; qb < SUB / 32; ++qb) {
        float p[16];
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
          const f32x4 l4 = *(const f32x4*)(&lse_s[rb][32 * qb + 8 * grp + 4 * hi]);
#pragma unroll
          for (int e = 0; e < 4; ++e) p[4 * grp + e] = fast_exp2(__builtin_fmaf(sp[qb][4 * grp + e], a.scale_log2, -l4[e]));
        }
        if (masked) {
#pragma unroll
          for (int grp = 0; grp < 4; ++grp) {
            const int q4 = 32 * qb + 8 * grp + 4 * hi;
            const i32x4 s4 = *(const i32x4*)(&start_s[rb][q4]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if ((uint32_t)(gk - s4[e]) > (uint32_t)(gq0 + q4 + e - s4[e])) p[4 * grp + e] = 0.f;
          }
        }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          h16x8 ph;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const auto pk = __builtin_amdgcn_cvt_pkrtz(p[8 * half + 2 * i], p[8 * half + 2 * i + 1]);
            ph[2 * i] = pk[0];
            ph[2 * i + 1] = pk[1];
          }
          Px[pbuf][kb][qb][half][lane] = ph;
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) opnd[qb][j >> 3][j & 7] = (__bf16)p[j];
      }
    }
  };
  // Gradient products of a sub-tile (buffer tb): dV += P^T dO (S wave, dO read transposed) or
  // dS = P (dP - delta), dK += dS^T Q (dP wave, P from the hand-off, Q read transposed)
  auto products = [&](int tb, int pbuf) {
    const __bf16* T = s_wave ? dOs[tb] : Qs[tb];
#pragma unroll
    for (int qb = 0; qb < SUB / 32; ++qb) {
      bf16x8 bt[2][MB];  // 16 queries per MFMA
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int rb = (32 * qb + 16 * half) * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          bt[half][mb] = cat4(ds_read_tr16(T + rb + troff[mb][0]), ds_read_tr16(T + rb + 8 * D + troff[mb][1]));
      }
      if (!s_wave) {
        // dS = P (dP - delta): one mixed-precision multiply per element (fp16 P, fp32 dP - delta)
        const h16x8 ph[2] = {Px[pbuf][kb][qb][0][lane], Px[pbuf][kb][qb][1][lane]};
#pragma unroll
        for (int j = 0; j < 16; ++j)
          opnd[qb][j >> 3][j & 7] = (__bf16)__builtin_fmaf((float)ph[j >> 3][j & 7], sp[qb][j], 0.f);
      }
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma32(opnd[qb][half], bt[half][mb], acc[mb]);
    }
  };
  auto sub_mask = [&](const Pos& p, bool& masked, int32_t& gq0) {
    const uint32_t t = tile_at(p);
    masked = (t >> 31) != 0;
    gq0 = (int32_t)global_pos(a.geom, a.shard, q0_at(t, p));
  };

  // prologue: sub-tiles 0 and 1 staged, the scores of sub-tile 0
  Pos cur{0, 0, 0};
  Pos nx1 = advance(cur);
  bool m0;
  int32_t g0;
  sub_mask(cur, m0, g0);
  load_sub(cur, 0);
  store_sub(0);
  if (total > 1) {
    load_sub(nx1, 1);
    store_sub(1);
  }
  // The compiler does not see the waits inside asm statements: without a use of the K (or V) rows
  // here it would wait for their loads at their first use inside the loop, in every iteration,
  // and since the counter also counts the transfers, each iteration would wait for the next
  // sub-tiles before its first product.
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) asm volatile("" ::"v"(kv[kk]));
  asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  scores(0, 0, m0, g0);
  hsap_lds_barrier();  // P of sub-tile 0 is in LDS

  // Iteration t: the gradient products of sub-tile t, then the scores of sub-tile t + 1, while
  // sub-tile t + 2 is moved into the third buffer; one barrier.  Both waves of a SIMD start with
  // independent work (the S wave's products on P it holds, the dP wave's dS arithmetic) and the S
  // wave's exponentials follow its score products while the dP wave's products run.
  int b0 = 0;  // t % 3
  for (int t = 0; t < total; ++t) {
    const int b1 = b0 == 2 ? 0 : b0 + 1, b2 = b1 == 2 ? 0 : b1 + 1;
    const Pos nx2 = advance(nx1);
    bool m1 = false;
    int32_t g1 = 0;
    if (t + 1 < total) sub_mask(nx1, m1, g1);  // before the window of t + 2 may replace it
    if (t + 2 < total) load_sub(nx2, b2);       // buffer b2 was last read before the previous barrier
    products(b0, t & 1);
    if (t + 1 < total) scores(b1, (t + 1) & 1, m1, g1);
    if (t + 2 < total) store_sub(b2);
    // sub-tile t + 2 has landed and is staged; P of t + 1 is in LDS; buffer b0 is free
    asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    nx1 = nx2;
    b0 = b1;
  }

  // this workgroup owns rows [krow0, krow0 + 128) of chunk c for K/V head g: the S waves write dV,
  // the dP waves dK (scaled)
  const float mul = s_wave ? 1.f : a.scale;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t idx = ((kvrow + 32 * kb + c_row(j, hi)) * a.hkv + g) * D + 32 * mb + l32;
      const float val = acc[mb][j] * mul;
      if (BF16OUT) {
        (s_wave ? a.dv16 : a.dk16)[idx] = (__bf16)val;
      } else {
        float* dst = s_wave ? a.dv : a.dk;
        dst[idx] += val;
      }
    }
}

// ---------------------------------------------------------------------------
// dQ kernel: one workgroup per (q-major run, query head), shaped like the
// forward.  Wave w owns 32 query rows; in the transposed orientation
// S^T = K Q^T and dP^T = V dO^T a lane holds one query, so its LSE and delta
// are scalars of the lane.  Per step of 64 keys:
//   P^T = exp2(S^T * scale*log2e - LSE*log2e), dS^T = P^T o (dP^T - delta),
//   dQ^T += K^T dS^T (K^T read transposed from the [key][d] tile).
// A run may span several chunks (tile by tile), so one run per q-tile covers
// every chunk; dQ stays in registers for the whole run and is written once at
// the end, by the q-tile's only run: a plain read-add-write of the fp32
// accumulator, or a store of the final bf16 value.
// ---------------------------------------------------------------------------
template <int D, int BN, int WAVES, bool BF16OUT, bool LIST = false>
__global__ __launch_bounds__(64 * WAVES, 2) void attn_bwd_dq_kernel(BwdArgs a) {
  static_assert(!LIST || !BF16OUT, "the tile-list mode accumulates fp32");
  constexpr int KB = 64;                     // keys per step
  constexpr int SUBS = BN / KB;
  constexpr int NT = 64 * WAVES;
  constexpr int CPR = D / 8;
  constexpr int MB = D / 32;
  constexpr int CHUNKS = KB * CPR;           // 16-byte chunks per K (or V) step
  static_assert(CHUNKS % NT == 0, "step must split evenly over the threads");
  constexpr float LOG2E = 1.44269504088896340736f;
  constexpr float NEG_INF = -__builtin_inff();
  __shared__ __attribute__((aligned(16))) __bf16 Ks[2][KB * D];  // swizzled [key][d]
  __shared__ __attribute__((aligned(16))) __bf16 Vs[2][KB * D];

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  int run_idx, h;
  run_and_head(blockIdx.x, a.hq, a.hkv, run_idx, h);
  // LIST: the tile-list mode, this workgroup's q-tile found in one chunk's list
  const hsap_run run = LIST ? q_tile_run(a.tiles, a.num_tiles, run_idx, lane) : a.runs[run_idx];
  const int g = h / a.group;
  const int64_t n = a.geom.n;
  const int64_t qrow = (int64_t)run.tile * (32 * WAVES) + 32 * w + l32;
  if (run.count == 0) {  // no key for this q-tile: dQ = 0
    if (BF16OUT) {
      bf16x4* dst = (bf16x4*)(a.dq16 + (qrow * a.hq + h) * D + 4 * hi);
#pragma unroll
      for (int e = 0; e < D / 8; ++e) dst[2 * e] = bf16x4{};
    }
    return;
  }
  const int32_t gq = (int32_t)global_pos(a.geom, a.shard, qrow);
  const int32_t qstart = a.doc_start[gq];
  const uint32_t span = (uint32_t)(gq - qstart);
  const float lse_raw = a.lse[(int64_t)h * n + qrow];
  const float lse2 = lse_raw == NEG_INF ? __builtin_inff() : lse_raw * LOG2E;  // no key: P = 0
  bf16x8 qf[D / 16], of[D / 16];
  float dlt;
  {
    const int64_t off = (qrow * a.hq + h) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      qf[kk] = *(const bf16x8*)(a.q + off + 16 * kk);
      of[kk] = *(const bf16x8*)(a.d_o + off + 16 * kk);
    }
    if (a.o) {
      // the backward preprocess for this row, delta = sum_d dO O, summed in the order of
      // hsap_attn_bwd_preprocess (so both give the same bits): a sum per 8-element chunk, then a
      // tree over the chunk index from its highest bit down.  The lane holds chunks 2 kk + hi, so
      // the tree runs over kk within the lane and ends with the lane l ^ 32 (chunk bit 0).
      float p[D / 16];
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) {
        const bf16x8 ov = *(const bf16x8*)(a.o + off + 16 * kk);
        p[kk] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) p[kk] = __builtin_fmaf((float)ov[e], (float)of[kk][e], p[kk]);
      }
#pragma unroll
      for (int wdt = D / 32; wdt >= 1; wdt >>= 1)
#pragma unroll
        for (int kk = 0; kk < wdt; ++kk) p[kk] = p[kk] + p[kk + wdt];
      dlt = p[0] + __shfl_xor(p[0], 32);
      if (hi == 0) a.delta_out[(int64_t)h * n + qrow] = dlt;  // read by the dK/dV kernel, launched after
    } else {
      dlt = a.delta[(int64_t)h * n + qrow];
    }
  }
  f32x16 ndlt;
#pragma unroll
  for (int j = 0; j < 16; ++j) ndlt[j] = -dlt;
  const int tr_row = 4 * hi + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int rowoff[D / 16], troff[MB][2];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) rowoff[kk] = swz<CPR>(l32, 16 * kk + 8 * hi);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int k = 0; k < 2; ++k) troff[mb][k] = swz<CPR>(8 * k + tr_row, 32 * mb + tr_col) - 8 * k * D;

  const int64_t rstride = (int64_t)a.hkv * D;
  const int total = run.count * SUBS;
  // The run's tile descriptors, packed one per lane (k_tile | chunk << 23 | kind << 31) in windows
  // of 64 tiles (window v in win0 or win1 by parity), read with v_readlane: the loop issues no
  // vector load besides the transfers (one would wait for every transfer in flight).
  uint32_t win0 = 0u, win1 = 0u;
  int win_hi = -1;
  auto load_window = [&](int v) {
    const int i = 64 * v + lane;
    uint32_t p = 0;
    if (i < run.count) {
      const hsap_tile t = a.tiles[run.first + i];
      p = (uint32_t)t.k_tile | ((uint32_t)t.chunk << 23) | ((uint32_t)t.kind << 31);
    }
    if (v & 1) win1 = p;
    else win0 = p;
    win_hi = v;
  };
  auto tile_at = [&](int s) -> uint32_t {
    const int idx = s / SUBS;
    return __builtin_amdgcn_readlane(((idx >> 6) & 1) ? win1 : win0, idx & 63);
  };
  auto chunk_of = [](uint32_t p) { return (int32_t)((p >> 23) & 0xFFu); };
  auto step_row0 = [&](uint32_t p, int s) { return (int64_t)(p & 0x7FFFFFu) * BN + (s % SUBS) * KB; };
  // the step's first row in the sharded K/V buffers: chunk of the tile, K/V head g
  auto step_off = [&](uint32_t p, int s) { return (((int64_t)chunk_of(p) * n + step_row0(p, s)) * a.hkv + g) * D; };
  load_window(0);

  // K and V steps go from global memory straight into LDS (global_load_lds) in a two-slot ring of
  // swizzled tiles: the next step's transfers are issued at the start of a step into the slot the
  // previous step read, and have landed at the step's closing barrier.  Instruction u of wave w
  // fills chunk positions p = WCH w + 64 u + lane; the lane's source is the chunk the swizzle
  // places there, a 32-bit byte offset from the step's scalar base.
  constexpr int WCH = CHUNKS / WAVES, U = WCH / 64;
  static_assert(WCH % 64 == 0, "a wave moves whole instructions of a tile");
  uint32_t gsrc[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int p = WCH * w + 64 * u + lane, row = p / CPR;
    gsrc[u] = (uint32_t)((row * rstride + swz_chunk<CPR>(row, p % CPR) * 8) * 2);
  }
  typedef __attribute__((address_space(3))) void* lds_void;
  const int wu = __builtin_amdgcn_readfirstlane(w);
  auto stage = [&](const __bf16* src, __bf16* dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_void)dst + (uint32_t)(WCH * wu * 16);
#pragma unroll
    for (int u = 0; u < U; ++u)
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(gsrc[u]), "s"(src), "{m0}"(lds + 64 * 16 * u));
  };

  f32x16 dq[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) dq[mb] = f32x16{};

  {
    const int64_t off = step_off(tile_at(0), 0);
    stage(a.k + off, Ks[0]);
    stage(a.v + off, Vs[0]);
  }
  // The compiler does not see the waits inside asm statements: without a use of Q and dO here it
  // would wait for their loads at their first use inside the loop, in every step, and since the
  // counter also counts the step's transfers, each step would wait for the next step's K and V.
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) asm volatile("" ::"v"(qf[kk]), "v"(of[kk]));
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");

  // one 64-key step from slot PAR (= s % 2, a compile-time constant, so every slot address is an
  // immediate); the next step's transfers go to the other slot
  auto step = [&](int s, auto par) __attribute__((always_inline)) {
    constexpr int PAR = decltype(par)::value;
    if (s + 1 < total && ((s + 1) / SUBS) >> 6 > win_hi) load_window(win_hi + 1);
    const uint32_t tile = tile_at(s);
    if (s + 1 < total) {
      const int64_t off = step_off(tile_at(s + 1), s + 1);
      stage(a.k + off, Ks[PAR ^ 1]);
      stage(a.v + off, Vs[PAR ^ 1]);
    }
    const __bf16* K = Ks[PAR];
    const __bf16* V = Vs[PAR];
    // Masked tile: a step whose keys no query of the wave may see contributes nothing (skipped);
    // one whose keys every query of the wave may see needs no per-element mask.
    bool live = true, need_mask = false;
    int32_t rel0 = 0;  // key row of register j: rel0 + 32 nb + c_row(j, 0)
    if (tile >> 31) {
      const int32_t r = (int32_t)global_pos(a.geom, chunk_of(tile), step_row0(tile, s)) - qstart;
      const bool none = r > (int32_t)span || r + (KB - 1) < 0;
      const bool all = r >= 0 && r + (KB - 1) <= (int32_t)span;
      live = __builtin_amdgcn_ballot_w64(!none) != 0;
      need_mask = live && __builtin_amdgcn_ballot_w64(!all) != 0;
      rel0 = r + 4 * hi;
    }
    if (live) {
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb) {
        // dP^T accumulates onto -delta (ndlt), so the chain ends with dP^T - delta
        f32x16 st{}, dpt = ndlt;
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          st = mfma32(*(const bf16x8*)(K + 32 * nb * D + rowoff[kk]), qf[kk], st);
          dpt = mfma32(*(const bf16x8*)(V + 32 * nb * D + rowoff[kk]), of[kk], dpt);
        }
        float p[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) p[j] = fast_exp2(__builtin_fmaf(st[j], a.scale_log2, -lse2));
        if (need_mask) {  // uniform branch: the mask costs nothing on steps that need none
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if ((uint32_t)(rel0 + (32 * nb + c_row(j, 0))) > span) p[j] = 0.f;
        }
        bf16x8 sb[2];
#pragma unroll
        for (int j = 0; j < 16; ++j) sb[j >> 3][j & 7] = (__bf16)(p[j] * dpt[j]);
        // dQ^T += K^T dS^T, 16 keys per MFMA
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int rb = (32 * nb + 16 * half) * D;
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            const bf16x8 ka = cat4(ds_read_tr16(K + rb + troff[mb][0]), ds_read_tr16(K + rb + 8 * D + troff[mb][1]));
            dq[mb] = mfma32(ka, sb[half], dq[mb]);
          }
        }
      }
    }
    // every read of slot PAR is done and the transfers into slot PAR ^ 1 have landed
    asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  for (int s = 0; s < total; s += 2) {
    step(s, std::integral_constant<int, 0>{});
    if (s + 1 < total) step(s + 1, std::integral_constant<int, 1>{});
  }

  // dQ^T: this lane's query, d = 32 mb + 8 grp + 4 hi + e for register j = 4 grp + e
  const int64_t base = (qrow * a.hq + h) * D + 4 * hi;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const f32x4 val{dq[mb][4 * grp] * a.scale, dq[mb][4 * grp + 1] * a.scale, dq[mb][4 * grp + 2] * a.scale,
                      dq[mb][4 * grp + 3] * a.scale};
      if (BF16OUT) {
        *(bf16x4*)(a.dq16 + base + 32 * mb + 8 * grp) = bf16x4{(__bf16)val[0], (__bf16)val[1], (__bf16)val[2],
                                                               (__bf16)val[3]};
      } else {
        f32x4* dst = (f32x4*)(a.dq + base + 32 * mb + 8 * grp);
        *dst = *dst + val;
      }
    }
}

template <int D, int WAVES, bool BF16OUT, bool LIST = false>
static hsap_status launch_dkdv(const BwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hkv;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, WAVES, BF16OUT, LIST>), dim3((unsigned)blocks), dim3(64 * WAVES), 0,
                     stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_bwd_dkdv launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

template <bool BF16OUT>
static hsap_status launch_dkdv_split(const BwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hkv;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  hipLaunchKernelGGL((attn_bwd_dkdv_split_kernel<BF16OUT>), dim3((unsigned)blocks), dim3(512), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_bwd_dkdv_split launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

template <int D, int BN, int WAVES, bool BF16OUT, bool LIST = false>
static hsap_status launch_dq(const BwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hq;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, BN, WAVES, BF16OUT, LIST>), dim3((unsigned)blocks), dim3(64 * WAVES), 0,
                     stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_bwd_dq launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}


// Packed tile descriptors of the dQ kernel: chunks below 256, k-tiles below 2^23.
constexpr int kMaxDqChunks = 256;
constexpr int64_t kMaxDqKTiles = int64_t(1) << 23;

}  // namespace hsap

// (head_dim, BM, BN) combinations with both backward kernels: the dK/dV kernel takes any BM that
// is a multiple of 64 (64-row sub-tiles) and BN = 32 x waves; the dQ kernel BM = 32 x waves.
bool hsap::backward_supported(const hsap_attn_desc* desc) {
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  const bool dkdv_ok = bm % 64 == 0 && ((d == 128 && (bn == 128 || bn == 64)) || (d == 64 && bn == 64));
  const bool dq_ok = (bm == 128 || bm == 64 || (bm == 256 && d == 128)) && (bn == 128 || bn == 64);
  return dkdv_ok && dq_ok;
}

namespace hsap {

// shared checks and dispatch of the fp32-accumulating and the bf16-storing backward
template <bool BF16OUT>
// o == NULL: delta is an input.  Otherwise the dQ kernel computes delta from o and d_o into
// delta_out, and the dK/dV kernel (launched after it) reads it there.
static hsap_status backward(const hsap_attn_desc* desc, const void* q, const void* k, const void* v, const void* d_o,
                            const void* o, const float* lse, const float* delta, float* delta_out,
                            const int32_t* doc_start, const hsap_tile* tiles_k, const hsap_run* runs_k,
                            int64_t num_runs_k, const hsap_tile* tiles_q, const hsap_run* runs_q,
                            int64_t num_runs_q, void* dq, void* dk, void* dv, hipStream_t s) {
  Geom geom;
  hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  if (num_runs_k < 0 || num_runs_q < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "negative run count");
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  if (!backward_supported(desc))
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no backward kernel for head_dim=%d BM=%d BN=%d", d, bm, bn);
  if ((int64_t)desc->heads_kv * d * 64 > INT32_MAX) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "heads_kv too large");
  // the dQ kernel packs a tile descriptor as k_tile | chunk << 23 | kind << 31
  if (num_runs_q > 0 && (geom.P > kMaxDqChunks || geom.n / bn >= kMaxDqKTiles))
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "the dQ kernel needs sp_degree <= %d and fewer than 2^23 k-tiles per chunk "
              "(sp_degree %d)", kMaxDqChunks, geom.P);
  if (num_runs_k == 0 && num_runs_q == 0) return HSAP_OK;
  if (!q || !k || !v || !d_o || !lse || !(o ? delta_out : delta) || !doc_start || !dq || !dk || !dv ||
      (num_runs_k > 0 && (!tiles_k || !runs_k)) || (num_runs_q > 0 && (!tiles_q || !runs_q)))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)d_o | (uintptr_t)o) & 15)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q, k, v, d_o and o must be 16-byte aligned");
  if (o && num_runs_k > 0 && num_runs_q == 0)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "delta from o needs the q-major runs (the dQ kernel computes it)");
  if ((uintptr_t)dq & (BF16OUT ? 7 : 15))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "dq must be %d-byte aligned", BF16OUT ? 8 : 16);
  BwdArgs a = {};
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.d_o = (const __bf16*)d_o;
  a.lse = lse;
  a.delta = o ? delta_out : delta;
  a.o = (const __bf16*)o;
  a.delta_out = delta_out;
  a.doc_start = doc_start;
  if (BF16OUT) {
    a.dq16 = (__bf16*)dq;
    a.dk16 = (__bf16*)dk;
    a.dv16 = (__bf16*)dv;
  } else {
    a.dq = (float*)dq;
    a.dk = (float*)dk;
    a.dv = (float*)dv;
  }
  a.geom = geom;
  a.shard = desc->shard.shard_id;
  a.hq = desc->heads_q;
  a.hkv = desc->heads_kv;
  a.group = desc->heads_q / desc->heads_kv;
  a.bm = bm;
  a.scale = desc->softmax_scale;
  a.scale_log2 = desc->softmax_scale * 1.44269504088896340736f;
  if (num_runs_q > 0) {
    a.tiles = tiles_q;
    a.runs = runs_q;
#define HSAP_DQ_CASE(D_, BN_, W_) \
  if (d == D_ && bn == BN_ && bm == 32 * W_) st = launch_dq<D_, BN_, W_, BF16OUT>(a, num_runs_q, s);
    HSAP_DQ_CASE(128, 128, 8)
    else HSAP_DQ_CASE(128, 64, 8)
    else HSAP_DQ_CASE(128, 128, 4)
    else HSAP_DQ_CASE(128, 64, 4)
    else HSAP_DQ_CASE(128, 128, 2)
    else HSAP_DQ_CASE(128, 64, 2)
    else HSAP_DQ_CASE(64, 128, 4)
    else HSAP_DQ_CASE(64, 64, 4)
    else HSAP_DQ_CASE(64, 128, 2)
    else HSAP_DQ_CASE(64, 64, 2)
#undef HSAP_DQ_CASE
    if (st != HSAP_OK) return st;
    a.o = nullptr;  // the dK/dV kernel reads delta
  }
  if (num_runs_k > 0) {
    a.tiles = tiles_k;
    a.runs = runs_k;
    if (d == 128 && bn == 128) st = launch_dkdv_split<BF16OUT>(a, num_runs_k, s);
    else if (d == 128) st = launch_dkdv<128, 2, BF16OUT>(a, num_runs_k, s);
    else st = launch_dkdv<64, 2, BF16OUT>(a, num_runs_k, s);
    if (st != HSAP_OK) return st;
  }
  return HSAP_OK;
}

// hsap_partial_attn_bwd: both kernels in tile-list mode over one chunk's tiles (fp32 accumulators).
static hsap_status backward_tile_list(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                      const void* d_o, const float* lse, const float* delta,
                                      const int32_t* doc_start, const hsap_tile* tiles, int64_t num_tiles,
                                      float* dq, float* dk, float* dv, hipStream_t s) {
  Geom geom;
  hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  if (!backward_supported(desc))
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no backward kernel for head_dim=%d BM=%d BN=%d", d, bm, bn);
  if ((int64_t)desc->heads_kv * d * 64 > INT32_MAX) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "heads_kv too large");
  if (desc->chunk_id < 0 || desc->chunk_id >= geom.P)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "chunk_id %d outside [0, %d)", desc->chunk_id, geom.P);
  if (num_tiles < 0 || num_tiles > (int64_t(1) << 30))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad num_tiles %lld", (long long)num_tiles);
  if (geom.n / bm > kMaxListQTiles)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "the tile-list backward needs n / BM <= %d (%lld)", kMaxListQTiles,
              (long long)(geom.n / bm));
  if (geom.n / bn >= kMaxDqKTiles) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "too many k-tiles per chunk");
  if (!q || !k || !v || !d_o || !lse || !delta || !doc_start || !dq || !dk || !dv || (num_tiles > 0 && !tiles))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)d_o | (uintptr_t)dq) & 15)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q, k, v, d_o and dq_acc must be 16-byte aligned");
  if (num_tiles == 0) return HSAP_OK;  // no pair of this shard and chunk: every gradient term is 0
  BwdArgs a = {};
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.d_o = (const __bf16*)d_o;
  a.lse = lse;
  a.delta = delta;
  a.doc_start = doc_start;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.geom = geom;
  a.shard = desc->shard.shard_id;
  a.hq = desc->heads_q;
  a.hkv = desc->heads_kv;
  a.group = desc->heads_q / desc->heads_kv;
  a.bm = bm;
  a.scale = desc->softmax_scale;
  a.scale_log2 = desc->softmax_scale * 1.44269504088896340736f;
  a.tiles = tiles;
  a.runs = nullptr;
  a.num_tiles = (int32_t)num_tiles;
  a.chunk = desc->chunk_id;
  const int64_t q_tiles = geom.n / bm, k_tiles = geom.n / bn;
#define HSAP_DQ_CASE(D_, BN_, W_) \
  if (d == D_ && bn == BN_ && bm == 32 * W_) st = launch_dq<D_, BN_, W_, false, true>(a, q_tiles, s);
  HSAP_DQ_CASE(128, 128, 8)
  else HSAP_DQ_CASE(128, 64, 8)
  else HSAP_DQ_CASE(128, 128, 4)
  else HSAP_DQ_CASE(128, 64, 4)
  else HSAP_DQ_CASE(128, 128, 2)
  else HSAP_DQ_CASE(128, 64, 2)
  else HSAP_DQ_CASE(64, 128, 4)
  else HSAP_DQ_CASE(64, 64, 4)
  else HSAP_DQ_CASE(64, 128, 2)
  else HSAP_DQ_CASE(64, 64, 2)
#undef HSAP_DQ_CASE
  if (st != HSAP_OK) return st;
  if (d == 128 && bn == 128) return launch_dkdv<128, 4, false, true>(a, k_tiles, s);
  if (d == 128) return launch_dkdv<128, 2, false, true>(a, k_tiles, s);
  return launch_dkdv<64, 2, false, true>(a, k_tiles, s);
}

}  // namespace hsap

using namespace hsap;

extern "C" hsap_status hsap_partial_attn_bwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const void* d_o, const float* lse, const float* delta,
                                             const int32_t* doc_start, const hsap_tile* tiles, int64_t num_tiles,
                                             float* dq_acc, float* dk_acc, float* dv_acc, void* hip_stream) {
  clear_error();
  return backward_tile_list(desc, q, k, v, d_o, lse, delta, doc_start, tiles, num_tiles, dq_acc, dk_acc, dv_acc,
                            (hipStream_t)hip_stream);
}

extern "C" hsap_status hsap_partial_attn_bwd_runs(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const void* d_o, const float* lse, const float* delta,
                                             const int32_t* doc_start, const hsap_tile* tiles_k,
                                             const hsap_run* runs_k, int64_t num_runs_k, const hsap_tile* tiles_q,
                                             const hsap_run* runs_q, int64_t num_runs_q, float* dq_acc,
                                             float* dk_acc, float* dv_acc, void* hip_stream) {
  clear_error();
  return backward<false>(desc, q, k, v, d_o, nullptr, lse, delta, nullptr, doc_start, tiles_k, runs_k, num_runs_k,
                         tiles_q, runs_q, num_runs_q, dq_acc, dk_acc, dv_acc, (hipStream_t)hip_stream);
}

extern "C" hsap_status hsap_attn_bwd_bf16(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                          const void* d_o, const float* lse, const float* delta,
                                          const int32_t* doc_start, const hsap_tile* tiles_k, const hsap_run* runs_k,
                                          int64_t num_runs_k, const hsap_tile* tiles_q, const hsap_run* runs_q,
                                          int64_t num_runs_q, void* dq, void* dk, void* dv, void* hip_stream) {
  clear_error();
  return backward<true>(desc, q, k, v, d_o, nullptr, lse, delta, nullptr, doc_start, tiles_k, runs_k, num_runs_k,
                        tiles_q, runs_q, num_runs_q, dq, dk, dv, (hipStream_t)hip_stream);
}

namespace hsap {
hsap_status attn_bwd_bf16_delta(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                const void* d_o, const void* o, const float* lse, float* delta,
                                const int32_t* doc_start, const hsap_tile* tiles_k, const hsap_run* runs_k,
                                int64_t num_runs_k, const hsap_tile* tiles_q, const hsap_run* runs_q,
                                int64_t num_runs_q, void* dq, void* dk, void* dv, hipStream_t stream) {
  if (!o) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL o");
  return backward<true>(desc, q, k, v, d_o, o, lse, nullptr, delta, doc_start, tiles_k, runs_k, num_runs_k, tiles_q,
                        runs_q, num_runs_q, dq, dk, dv, stream);
}
}  // namespace hsap
