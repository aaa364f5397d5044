// Partial attention forward: one shard's queries against the listed k-tiles of
// each K/V chunk ("computing" in the instruction table of the SAP section; the
// attention equation of the inter-group SP section under the packing mask).
//
// Work decomposition: one workgroup per (run, query head).  A run is one
// q-tile against some listed k-tiles of one chunk, written to its own
// partial slot (a long run may be split into several).  The workgroup has WAVES waves;
// wave w owns 32 query rows, so BM = 32 * WAVES.  Every listed k-tile of BN
// keys is consumed in steps of KB = 64 keys.
//
// Per step the workgroup stages the step's K and V rows in LDS, both in their
// natural [key][d] layout with 16-byte stores, and each wave computes the
// scores transposed, S^T = K Q^T, with Q held in registers as the MFMA B
// operand.  In that orientation a lane holds one query (its column) and 16
// keys per 32-key block, so the row max and row sum of the online softmax
// need only the lane and lane l ^ 32 (one permlane32 swap).  P (bf16) then
// feeds O^T += V^T P^T as the B operand straight from registers; the V^T
// operand is read from the [key][d] tile with the LDS transpose read, whose
// per-lane key order matches the register order of the score block.
//
// Pipelining: the scores of step s + 1 are computed on the matrix cores while
// the vector units run the softmax of step s.  K and V each have two LDS
// slots; the next K/V rows load into registers during a step and are written
// to the free slots at its end, one barrier per step.
// Scores are scaled by softmax_scale * log2(e) so the exponentials are exp2.
// FULL tiles skip all mask arithmetic; MASKED tiles compare each key position
// with the query's document start and position.  O is rescaled only when
// some row of the wave raised its running max by more than a fixed slack.
#include <type_traits>

#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

// Third word of a raw buffer descriptor on gfx9-family targets (32-bit data format; the format
// is ignored by untyped loads, but a zero format makes them return zeros).
constexpr int kBufferWord3 = 0x00020000;

// The direct-to-LDS kernel packs a tile descriptor as k_tile | chunk << 23 | kind << 31.
constexpr int kMaxDlChunks = 256;
constexpr int64_t kMaxDlKTiles = int64_t(1) << 23;

struct FwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const int32_t* doc_start;
  const hsap_tile* tiles;
  const hsap_run* runs;
  float* o_part;
  float* lse_part;
  int32_t num_slots;
  __bf16* o_out;    // fused forward: final output [n, Hq, d]
  float* lse_out;   // fused forward: final LSE [Hq, n]
  const float* q_scale;  // fp8 scores: dequantisation scale per query head [Hq]
  const float* k_scale;  // fp8 scores: dequantisation scale per (chunk, K/V head) [P, Hkv]
  const int32_t* cu;     // when set: cumulative document lengths [num_docs + 1], used instead of doc_start
  int32_t num_docs;
  int32_t num_tiles;     // runs == NULL: one chunk's tiles sorted by q_tile; workgroup t runs q-tile t
  Geom geom;
  int32_t shard;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  float scale_log2;
};

// Document start of this lane's query (global position gq), in two parts so the memory access
// is issued at kernel start and consumed after the prologue.  With per-position starts it is one
// load.  From the cumulative lengths instead: a wave's 32 queries (lanes 0..31; lane l ^ 32 holds
// the query of lane l) are 32 consecutive positions -- every piece of a shard is a multiple of
// the 64-, 128- or 256-row q-tile -- so at most 31 document boundaries lie after the document of
// lane 0's position g_lo, up to lane 31's position g_hi.  The wave loads 64 consecutive entries
// of cu_seqlens, starting at most 31 entries before the document of g_lo (a 64-way search in
// rounds narrows the start when there are more than 32 entries), and each lane takes the largest
// entry not above its position with ballots and lane reads: no further memory access.
struct DocWindow {
  int32_t w;           // cu[base + lane], or this lane's start when per-position starts are given
  int32_t g_lo, g_hi;  // positions of the wave's first and last query
};

__device__ __forceinline__ DocWindow doc_window(const FwdArgs& a, int32_t gq, int lane) {
  DocWindow r{};
  if (!a.cu) {
    r.w = a.doc_start[gq];
    return r;
  }
  r.g_lo = __builtin_amdgcn_readlane(gq, 0);
  r.g_hi = __builtin_amdgcn_readlane(gq, 31);
  const int32_t nd = a.num_docs;
  int32_t base = 0, len = nd + 1;  // the document of g_lo is one of base .. base + len - 1
  while (len > 32) {
    const int32_t stride = (len + 63) >> 6;
    const int32_t v = a.cu[min(base + lane * stride, nd)];
    base += stride * (__popcll(__builtin_amdgcn_ballot_w64(v <= r.g_lo)) - 1);
    len = stride;
  }
  r.w = a.cu[min(base + lane, nd)];
  return r;
}

__device__ __forceinline__ int32_t doc_window_start(const FwdArgs& a, const DocWindow& r, int32_t gq) {
  if (!a.cu) return r.w;
  const int32_t lo = __popcll(__builtin_amdgcn_ballot_w64(r.w <= r.g_lo)) - 1;    // document of g_lo
  const int32_t last = __popcll(__builtin_amdgcn_ballot_w64(r.w <= r.g_hi)) - 1;  // last boundary <= g_hi
  int32_t start = __builtin_amdgcn_readlane(r.w, lo);
  if (last >= 63) {  // more boundaries than the window holds (not reachable with validated shapes)
    int32_t l = 0, h = a.num_docs;
    while (h - l > 1) {
      const int32_t mid = (l + h) >> 1;
      if (a.cu[mid] <= gq) l = mid;
      else h = mid;
    }
    return a.cu[l];
  }
  for (int32_t j = lo + 1; j <= last; ++j) {
    const int32_t b = __builtin_amdgcn_readlane(r.w, j);
    if (gq >= b) start = b;
  }
  return start;
}

// fp8 scores: the exp2 scale of a step, q_scale[h] * k_scale[chunk, g] * scale * log2(e), kept at
// or above the smallest normal float.  A scale is 0 only when its slice is all zeros, so every
// code and every finite score of the step is 0 and stays 0 after the multiply, while a masked
// score (-inf) must stay -inf: times 0 it would turn into NaN and poison the row.
__device__ __forceinline__ float fp8_step_scale(float sl) { return fmaxf(sl, 1.17549435e-38f); }

// FP8: Q and K are e4m3 codes (scores S = (Q8 K8^T) * q_scale[h] * k_scale[chunk, g]
// from the 32x32x64 fp8 MFMA, a K row held as 128 bytes), V and the rest as in bf16.
template <int D, int BN, int WAVES, bool FUSED, bool FP8 = false, bool LIST = false>
__global__ __launch_bounds__(64 * WAVES, 2) void attn_fwd_kernel(FwdArgs a) {
  static_assert(!FP8 || D == 128, "fp8 scores need head_dim 128");
  static_assert(!LIST || (!FUSED && !FP8), "the tile-list mode is the bf16 partial forward's");
  using KT = std::conditional_t<FP8, uint8_t, __bf16>;    // K element
  using K16 = std::conditional_t<FP8, uint4, bf16x8>;     // 16 bytes of K
  constexpr int KB = 64;                     // keys per step
  constexpr int SUBS = BN / KB;              // steps per listed k-tile
  constexpr int NT = 64 * WAVES;
  // K row stride in elements: bf16 D + 8 (68 dwords), fp8 D + 16 (36 dwords); either way the
  // rows of a 16-lane b128 read hit distinct banks
  constexpr int KS = FP8 ? D + 16 : D + 8;
  constexpr int VS = D + 32;                 // V row stride (bf16): 16 (mod 64) dwords, 32 lanes of a transpose read hit distinct banks
  constexpr int CHUNKS = KB * D / 8;         // 16-byte chunks per V (and bf16 K) step
  constexpr int PER_T = CHUNKS / NT;         // chunks per thread
  constexpr int KCPR = D * (int)sizeof(KT) / 16;   // 16-byte chunks per K row
  constexpr int PER_TK = KB * KCPR / NT;     // K chunks per thread
  static_assert(CHUNKS % NT == 0 && (KB * KCPR) % NT == 0, "step must split evenly over the threads");
  constexpr float NEG_INF = -__builtin_inff();
  constexpr float RESCALE_SLACK = 8.f;       // log2 units a row max may rise before O is rescaled
  __shared__ __attribute__((aligned(16))) KT Ks[2][KB * KS];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[2][KB * VS];

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  int run_idx, h;  // runs are longest first: long work starts first
  run_and_head(blockIdx.x, a.hq, a.hkv, run_idx, h);
  // LIST: the tile-list mode of the partial forward, this workgroup's q-tile found in one chunk's list
  const hsap_run run = LIST ? q_tile_run(a.tiles, a.num_tiles, run_idx, lane) : a.runs[run_idx];
  const int slot = run.slot;  // partial-output slot of this run (partial forward)
  // FUSED, or a partial run marked final (its q-tile's only part): write the final output
  const bool final_out = FUSED || (slot == kFinalSlot && a.o_out != nullptr);
  if (!final_out && (slot < 0 || slot >= a.num_slots)) return;
  const int g = h / a.group;
  const int64_t n = a.geom.n;
  const int64_t qrow = (int64_t)run.tile * (32 * WAVES) + 32 * w + l32;  // this lane's query row (shard-local)

  if (run.count == 0) {  // no key for this q-tile in this run
    if (final_out) {
      bf16x4* op = (bf16x4*)(a.o_out + (qrow * a.hq + h) * D + 4 * hi);
#pragma unroll
      for (int e = 0; e < D / 8; ++e) op[2 * e] = bf16x4{};
      if (hi == 0) a.lse_out[(int64_t)h * n + qrow] = NEG_INF;
    } else if (hi == 0) {
      a.lse_part[((int64_t)slot * a.hq + h) * n + qrow] = NEG_INF;
    }
    return;
  }

  const int32_t gq = (int32_t)global_pos(a.geom, a.shard, qrow);
  const DocWindow docw = doc_window(a, gq, lane);
  bf16x8 qf[D / 16];
  i32x8 qf8[2];  // fp8: lane half hi holds bytes 64 kk + 32 hi .. +31 of its query's row
  if constexpr (FP8) {
    const uint8_t* qp = (const uint8_t*)a.q + (qrow * a.hq + h) * D + 32 * hi;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const uint4 lo = *(const uint4*)(qp + 64 * kk), hi4 = *(const uint4*)(qp + 64 * kk + 16);
      qf8[kk] = i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi4.x, (int)hi4.y, (int)hi4.z, (int)hi4.w};
    }
  } else {
    const __bf16* qp = a.q + (qrow * a.hq + h) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
  }
  // exp2 argument scale of this head (fp8: times the per-chunk K scale each step)
  const float head_scale = FP8 ? a.scale_log2 * a.q_scale[h] : a.scale_log2;
  const int64_t rstride = (int64_t)a.hkv * D;
  const int total = run.count * SUBS;
  auto tile_at = [&](int s) { return a.tiles[run.first + s / SUBS]; };
  // first K/V row of step s of tile t in the sharded buffers (chunk t.chunk, head g)
  auto step_row0 = [&](const hsap_tile& t, int s) { return (int64_t)t.k_tile * BN + (s % SUBS) * KB; };
  // a partial run stays in one chunk, so its base is fixed; a fused run changes chunk between tiles
  const int64_t run_base = FUSED ? 0 : (((int64_t)a.tiles[run.first].chunk * n) * a.hkv + g) * D;
  auto step_off = [&](const hsap_tile& t, int s) {
    if (FUSED) return (((int64_t)t.chunk * n + step_row0(t, s)) * a.hkv + g) * D;
    return run_base + step_row0(t, s) * rstride;
  };

  // staging: thread t moves chunks t, t + NT, ... of a step's [KB][D] tile, i.e. one column chunk
  // of rows r0, r0 + ROWS, r0 + 2 ROWS, ...  The distance between a thread's chunks is the same
  // for every thread, so the loads are buffer loads over the step's rows: the lane's byte offset
  // (loop-invariant, one VGPR) plus a uniform offset per chunk (SGPR), no address arithmetic per
  // load; the LDS stores take the chunk distance as an immediate offset.  The descriptor spans
  // exactly the step's KB rows, so the hardware range check bounds every access.
  constexpr int EPC = 16 / (int)sizeof(KT);  // K elements per 16-byte chunk
  constexpr int VROWS = NT / (D / 8), KROWS = NT / KCPR;
  static_assert(NT % (D / 8) == 0 && NT % KCPR == 0, "a thread's chunks must share their column");
  const int gvo = (int)(((tid / (D / 8)) * rstride + (tid % (D / 8)) * 8) * 2);
  const int gko = (int)(((tid / KCPR) * rstride + (tid % KCPR) * EPC) * (int)sizeof(KT));
  const int lvo = (tid / (D / 8)) * VS + (tid % (D / 8)) * 8;
  const int lko = (tid / KCPR) * KS + (tid % KCPR) * EPC;
  const int step_bytes_k = (int)(KB * rstride * (int)sizeof(KT)), step_bytes_v = (int)(KB * rstride * 2);
  K16 kreg[PER_TK];
  bf16x8 vreg[PER_T];
  auto load_k = [&](int64_t off) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc((void*)((const KT*)a.k + off), (short)0, step_bytes_k, kBufferWord3);
#pragma unroll
    for (int i = 0; i < PER_TK; ++i)
      kreg[i] = __builtin_bit_cast(
          K16, __builtin_amdgcn_raw_buffer_load_b128(r, gko, (int)(i * KROWS * rstride * (int)sizeof(KT)), 0));
  };
  auto load_v = [&](int64_t off) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc((void*)(a.v + off), (short)0, step_bytes_v, kBufferWord3);
#pragma unroll
    for (int i = 0; i < PER_T; ++i)
      vreg[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, gvo, (int)(i * VROWS * rstride * 2), 0));
  };
  auto store_k = [&](int slot) {
#pragma unroll
    for (int i = 0; i < PER_TK; ++i) *(K16*)(&Ks[slot][lko + i * KROWS * KS]) = kreg[i];
  };
  auto store_v = [&](int slot) {
#pragma unroll
    for (int i = 0; i < PER_T; ++i) *(bf16x8*)(&Vs[slot][lvo + i * VROWS * VS]) = vreg[i];
  };
  // S^T = K Q^T for the two 32-key blocks of a step held in K slot `slot`
  auto scores = [&](int slot, f32x16 (&sc)[KB / 32]) {
    const KT* K = Ks[slot];
#pragma unroll
    for (int nb = 0; nb < KB / 32; ++nb) {
      sc[nb] = f32x16{};
      if constexpr (FP8) {
        // the K row's bytes 64 kk + 32 hi .. +31 pair with the same bytes of the query's row
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const uint8_t* kp = K + (32 * nb + l32) * KS + 64 * kk + 32 * hi;
          const uint4 lo = *(const uint4*)kp, hi4 = *(const uint4*)(kp + 16);
          const i32x8 kf{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi4.x, (int)hi4.y, (int)hi4.z, (int)hi4.w};
          sc[nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf, qf8[kk], sc[nb], 0, 0, 0, 127, 0, 127);
        }
      } else {
        bf16x8 kf[D / 16];
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) kf[kk] = *(const bf16x8*)(K + (32 * nb + l32) * KS + 16 * kk + 8 * hi);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) sc[nb] = mfma32(kf[kk], qf[kk], sc[nb]);
      }
    }
  };

  // transpose-read geometry for the V^T operand (see mfma.h): lane j of each
  // 16-lane group points at 4 consecutive d of key row (j / 4) of its group
  const int tr_row = 4 * hi + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  constexpr int MB_OUT = D / 32;
  float m_run = NEG_INF, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};

  // Software pipeline: iteration s takes the softmax of step s, the scores of
  // step s + 1 and the PV product of step s.  K runs two steps ahead of use
  // and V one, so slot s % 2 of K (last read for the scores of step s, in
  // iteration s - 1, or before the loop for s = 0) and slot (s + 1) % 2 of V
  // (last read in iteration s - 1) are free to refill during iteration s; one
  // barrier per iteration orders the refills against the next iteration's
  // reads.
  const hsap_tile t_first = tile_at(0);
  load_k(step_off(t_first, 0));
  store_k(0);
  load_v(step_off(t_first, 0));
  store_v(0);
  if (total > 1) {
    load_k(step_off(tile_at(1), 1));
    store_k(1);
  }
  __syncthreads();
  f32x16 sc[KB / 32];
  scores(0, sc);
  __syncthreads();  // every wave has read K slot 0 before iteration 0 refills it
  const int32_t qstart = doc_window_start(a, docw, gq);  // first needed by the masks of step 0
  const uint32_t span = (uint32_t)(gq - qstart);  // key j is allowed iff 0 <= j - start <= span

  // one 64-key step: softmax and PV of step s from `sc`, scores of step s + 1 into `sn`; the
  // loop below runs it twice per iteration with the two score arrays swapped (no copy)
  // (`par` is s % 2 as a compile-time constant, so every LDS slot address is an immediate)
  auto step = [&](int s, auto par, f32x16 (&sc)[KB / 32], f32x16 (&sn)[KB / 32]) __attribute__((always_inline)) {
    constexpr int PAR = decltype(par)::value;
    const hsap_tile tile = tile_at(s);
    const float sl = FP8 ? fp8_step_scale(head_scale * a.k_scale[tile.chunk * a.hkv + g]) : head_scale;
    if (s + 2 < total) load_k(step_off(tile_at(s + 2), s + 2));
    if (s + 1 < total) load_v(step_off(tile_at(s + 1), s + 1));
    // scores of the next step: independent of this step's softmax
    if (s + 1 < total) scores(PAR ^ 1, sn);

    // Masked tile: a step whose keys no query of the wave may see is skipped (all its
    // probabilities would be 0: the running max, sum and O stay as they are), and one whose keys
    // every query of the wave may see needs no per-element mask.
    bool live = true;
    if (tile.kind == HSAP_TILE_MASKED) {
      const int32_t r = (int32_t)global_pos(a.geom, tile.chunk, step_row0(tile, s)) - qstart;  // offset of key 0
      const bool none = r > (int32_t)span || r + (KB - 1) < 0;
      const bool all = r >= 0 && r + (KB - 1) <= (int32_t)span;
      live = __builtin_amdgcn_ballot_w64(!none) != 0;
      if (live && __builtin_amdgcn_ballot_w64(!all) != 0) {
        // key row of register j: r + 32 nb + c_row(j, hi), with the lane's 4 hi folded in once
        const int32_t rel0 = r + 4 * hi;
#pragma unroll
        for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if ((uint32_t)(rel0 + (32 * nb + c_row(j, 0))) > span) sc[nb][j] = NEG_INF;
      }
    }
    if (live) {
      // online softmax (this lane's row = its query; lanes l and l ^ 32 share it)
      float mx = sc[0][0];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sc[nb][j]);
      const float m_new = fmaxf(m_run, pair_max(mx) * sl);
      // The reference max only has to bound the scores loosely: O / l and
      // m + log2(l) do not depend on it.  Rescale only when some row's max rose
      // by more than RESCALE_SLACK (p then stays below 2^RESCALE_SLACK).
      if (__builtin_amdgcn_ballot_w64(m_new > m_run + RESCALE_SLACK) != 0) {
        const float alpha = fast_exp2(m_run - (m_new == NEG_INF ? 0.f : m_new));
        l_run *= alpha;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
        m_run = m_new;
      }
      const float m_use = m_run == NEG_INF ? 0.f : m_run;
      float rs = 0.f;
      bf16x8 pb[KB / 32][2];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float p = fast_exp2(__builtin_fmaf(sc[nb][j], sl, -m_use));
          rs += p;
          pb[nb][j >> 3][j & 7] = (__bf16)p;
        }
      l_run += rs;  // the half-row sums of lanes l and l ^ 32 are combined once, at the end

      // O^T += V^T P^T, 16 keys per MFMA
      const __bf16* V = Vs[PAR];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int r0 = 32 * nb + 16 * half + tr_row;
#pragma unroll
          for (int mb = 0; mb < D / 32; ++mb) {
            const __bf16* vp = V + r0 * VS + 32 * mb + tr_col;
            const bf16x8 av = cat4(ds_read_tr16(vp), ds_read_tr16(vp + 8 * VS));
            o[mb] = mfma32(av, pb[nb][half], o[mb]);
          }
        }

    }
    if (s + 2 < total) store_k(PAR);
    if (s + 1 < total) store_v(PAR ^ 1);
    __syncthreads();
  };
  f32x16 sn[KB / 32];
  for (int s = 0; s < total; s += 2) {
    step(s, std::integral_constant<int, 0>{}, sc, sn);
    if (s + 1 < total) step(s + 1, std::integral_constant<int, 1>{}, sn, sc);
  }

  l_run = pair_sum(l_run);
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  const float lse = l_run > 0.f ? (m_run + __log2f(l_run)) * 0.69314718055994530942f : NEG_INF;
  if (final_out) {
    // final output: this lane's query, d = 32 mb + 8 grp + 4 hi + 0..3
    __bf16* op = a.o_out + (qrow * a.hq + h) * D + 4 * hi;
#pragma unroll
    for (int mb = 0; mb < MB_OUT; ++mb)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const bf16x4 val{(__bf16)(o[mb][4 * grp] * inv), (__bf16)(o[mb][4 * grp + 1] * inv),
                         (__bf16)(o[mb][4 * grp + 2] * inv), (__bf16)(o[mb][4 * grp + 3] * inv)};
        *(bf16x4*)(op + 32 * mb + 8 * grp) = val;
      }
    if (hi == 0) a.lse_out[(int64_t)h * n + qrow] = lse;
  } else {
    float* op = a.o_part + (((int64_t)slot * n + qrow) * a.hq + h) * D + 4 * hi;
#pragma unroll
    for (int mb = 0; mb < MB_OUT; ++mb)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const f32x4 val{o[mb][4 * grp] * inv, o[mb][4 * grp + 1] * inv, o[mb][4 * grp + 2] * inv,
                        o[mb][4 * grp + 3] * inv};
        *(f32x4*)(op + 32 * mb + 8 * grp) = val;
      }
    if (hi == 0) a.lse_part[((int64_t)slot * a.hq + h) * n + qrow] = lse;
  }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS forward for d = 128: WAVES waves (wave w owns query rows
// 32w..32w+31; BM = 32 WAVES).  K and V steps go from global memory straight
// into LDS (global_load_lds, no staging registers) in a ring of unpadded
// XOR-swizzled [64][128] tiles.  Eight waves (BM = 256, one workgroup per CU):
// three slots, K three steps ahead of its use in the scores and V two ahead of
// its use in PV, so a transfer has two steps to arrive.  Four waves (BM = 128,
// two workgroups per CU in 2 x 64 KB of LDS): two slots, K two steps ahead and
// V one, so a transfer has one step.  Each wave moves 1024 / WAVES of a tile's
// 1024 16-byte chunks, 64 per instruction; a lane's source chunk is the one
// the swizzle places at its destination.
//
// Order of a step: the step's transfers; the mask (MASKED tiles only), the
// row maximum and the rare rescale of O; then one straight-line block with
// the exponentials and PV of this step and the score products of the next,
// so that a wave's own vector work fills the shadow of its matrix products
// (scheduling-group barriers ask for that interleave).  The wave raises its
// priority for the block, so the SIMD's other wave (another workgroup) runs
// its transfers and row maximum meanwhile.  Every step forms the next
// step's scores; the last step's read a slot that no transfer is writing and
// are dropped.
// ---------------------------------------------------------------------------
// FP8: Q and K are e4m3 codes (scores from the 32x32x64 fp8 MFMA times q_scale[h] *
// k_scale[chunk, g]); K tiles are [64][128 bytes], swizzled over their 8 chunks per row.
template <int BN, int WAVES, bool FUSED, bool FP8 = false, bool LIST = false>
__global__ __launch_bounds__(64 * WAVES, 2) void attn_fwd_dl_kernel(FwdArgs a) {
  static_assert(WAVES == 4 || WAVES == 8, "four or eight waves");
  static_assert(!LIST || (!FUSED && !FP8), "the tile-list mode is the bf16 partial forward's");
  using KT = std::conditional_t<FP8, uint8_t, __bf16>;  // K element
  constexpr int D = 128, KB = 64, SUBS = BN / KB, CPR = D / 8, TILE = KB * D;
  constexpr int KCPR = D * (int)sizeof(KT) / 16;        // 16-byte chunks per K row
  constexpr int NSLOT = WAVES == 8 ? 3 : 2;  // ring depth
  constexpr int WCH = TILE / 8 / WAVES;      // 16-byte chunks of a V tile a wave moves
  constexpr int U = WCH / 64;                // transfer instructions per wave per V tile
  constexpr int WCHK = KB * KCPR / WAVES, UK = WCHK / 64;  // the same for a K tile
  static_assert(WCHK % 64 == 0, "a wave moves whole instructions of a K tile");
  constexpr float NEG_INF = -__builtin_inff();
  constexpr float RESCALE_SLACK = 8.f;
  __shared__ __attribute__((aligned(16))) KT Ks[NSLOT][TILE];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[NSLOT][TILE];
  __shared__ float kscale_s[FP8 ? kMaxDlChunks : 1];  // fp8: K scale of each chunk for this head's K/V head
  typedef __attribute__((address_space(3))) void* lds_void;

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  int run_idx, h;
  run_and_head(blockIdx.x, a.hq, a.hkv, run_idx, h);
  // LIST: the tile-list mode of the partial forward, this workgroup's q-tile found in one chunk's list
  const hsap_run run = LIST ? q_tile_run(a.tiles, a.num_tiles, run_idx, lane) : a.runs[run_idx];
  const int slot = run.slot;
  const bool final_out = FUSED || (slot == kFinalSlot && a.o_out != nullptr);
  if (!final_out && (slot < 0 || slot >= a.num_slots)) return;
  const int g = h / a.group;
  const int64_t n = a.geom.n;
  const int64_t qrow = (int64_t)run.tile * (32 * WAVES) + 32 * w + l32;

  if (run.count == 0) {
    if (final_out) {
      bf16x4* op = (bf16x4*)(a.o_out + (qrow * a.hq + h) * D + 4 * hi);
#pragma unroll
      for (int e = 0; e < D / 8; ++e) op[2 * e] = bf16x4{};
      if (hi == 0) a.lse_out[(int64_t)h * n + qrow] = NEG_INF;
    } else if (hi == 0) {
      a.lse_part[((int64_t)slot * a.hq + h) * n + qrow] = NEG_INF;
    }
    return;
  }

  const int32_t gq = (int32_t)global_pos(a.geom, a.shard, qrow);
  const DocWindow docw = doc_window(a, gq, lane);
  bf16x8 qf[D / 16];
  i32x8 qf8[2];  // fp8: lane half hi holds bytes 64 kk + 32 hi .. +31 of its query's row
  if constexpr (FP8) {
    const uint8_t* qp = (const uint8_t*)a.q + (qrow * a.hq + h) * D + 32 * hi;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const uint4 lo = *(const uint4*)(qp + 64 * kk), hi4 = *(const uint4*)(qp + 64 * kk + 16);
      qf8[kk] = i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi4.x, (int)hi4.y, (int)hi4.z, (int)hi4.w};
    }
  } else {
    const __bf16* qp = a.q + (qrow * a.hq + h) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
  }
  // exp2 argument scale of this head (fp8: times the chunk's K scale each step, from LDS, filled
  // here and visible after the prologue's barrier)
  const float head_scale = FP8 ? a.scale_log2 * a.q_scale[h] : a.scale_log2;
  if constexpr (FP8)
    for (int c = tid; c < a.geom.P; c += 64 * WAVES) kscale_s[c] = a.k_scale[c * a.hkv + (h / a.group)];
  const int64_t rstride = (int64_t)a.hkv * D;
  const int total = run.count * SUBS;
  // The run's tile descriptors, packed one per lane (k_tile | chunk << 23 | kind << 31) in
  // windows of 64 tiles (window v in win0 or win1 by parity), read with v_readlane: no memory
  // access for descriptors inside the loop (a vector load there would wait for every
  // transfer in flight).
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
  load_window(0);
  const int64_t run_base = FUSED ? 0 : (((int64_t)chunk_of(tile_at(0)) * n) * a.hkv + g) * D;
  auto step_off = [&](uint32_t p, int s) {
    if (FUSED) return (((int64_t)chunk_of(p) * n + step_row0(p, s)) * a.hkv + g) * D;
    return run_base + step_row0(p, s) * rstride;
  };

  // direct staging: instruction u of wave w fills chunk positions p = WCH w + 64 u + lane; the
  // lane's source is a 32-bit byte offset from the step's (scalar) base pointer
  uint32_t gsrc[U], gsrck[UK];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int p = WCH * w + 64 * u + lane, row = p >> 4;
    gsrc[u] = (uint32_t)((row * rstride + swz_chunk<CPR>(row, p & 15) * 8) * 2);
  }
#pragma unroll
  for (int u = 0; u < UK; ++u) {
    const int p = WCHK * w + 64 * u + lane, row = p / KCPR;
    gsrck[u] = (uint32_t)(row * rstride * (int)sizeof(KT) + swz_chunk<KCPR>(row, p % KCPR) * 16);
  }
  // issued from asm: the transfers are ordered by the explicit vmcnt waits of the ring below (the
  // compiler would otherwise wait for each one before any later LDS read).  No memory clobber:
  // volatile asm keeps its order against the ring's barriers (which do clobber memory), and the
  // tile descriptors stay scalar loads.
  // (M0, the LDS destination, is the slot's 32-bit LDS address plus the wave's chunk range: scalar
  // arithmetic only, with the wave index taken as uniform)
  const int wu = __builtin_amdgcn_readfirstlane(w);
  auto stage = [&](const __bf16* src, __bf16* dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_void)dst + (uint32_t)(WCH * wu * 16);
#pragma unroll
    for (int u = 0; u < U; ++u)
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(gsrc[u]), "s"(src), "{m0}"(lds + 64 * 16 * u));
  };
  auto stage_k = [&](const KT* src, KT* dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(lds_void)dst + (uint32_t)(WCHK * wu * 16);
#pragma unroll
    for (int u = 0; u < UK; ++u)
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(gsrck[u]), "s"(src), "{m0}"(lds + 64 * 16 * u));
  };
  const KT* kbase = (const KT*)a.k;

  // operand offsets in a swizzled tile: K rows (row l32 of a 32-row block, chunk 2 kk + hi) and
  // V transpose reads (rows 8 k + tr_row of a 16-row block, columns 32 mb + tr_col)
  const int tr_row = 4 * hi + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  int rowoff[D / 16], troff[D / 32][2];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) rowoff[kk] = swz<CPR>(l32, 16 * kk + 8 * hi);
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int k = 0; k < 2; ++k) troff[mb][k] = swz<CPR>(8 * k + tr_row, 32 * mb + tr_col) - 8 * k * D;

  // fp8 K reads: the K row's bytes 64 kk + 32 hi .. +31 (chunks 4 kk + 2 hi and the next) pair
  // with the same bytes of the query's row; byte offsets in the swizzled tile for row l32 (a
  // 32-row block further down keeps the swizzle)
  int koff8[2][2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int c = 0; c < 2; ++c) koff8[kk][c] = l32 * 128 + swz_chunk<8>(l32, 4 * kk + 2 * hi + c) * 16;
  auto scores = [&](const KT* K, f32x16 (&sc)[KB / 32]) {
#pragma unroll
    for (int nb = 0; nb < KB / 32; ++nb) {
      sc[nb] = f32x16{};
      if constexpr (FP8) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          const uint4 lo = *(const uint4*)(K + 32 * nb * 128 + koff8[kk][0]);
          const uint4 hi4 = *(const uint4*)(K + 32 * nb * 128 + koff8[kk][1]);
          const i32x8 kf{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi4.x, (int)hi4.y, (int)hi4.z, (int)hi4.w};
          sc[nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf, qf8[kk], sc[nb], 0, 0, 0, 127, 0, 127);
        }
      } else {
        bf16x8 kf[D / 16];
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) kf[kk] = *(const bf16x8*)(K + 32 * nb * D + rowoff[kk]);
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) sc[nb] = mfma32(kf[kk], qf[kk], sc[nb]);
      }
    }
  };

  float m_run = NEG_INF, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};

  // prologue: K(0 .. NSLOT - 1) and V(0 .. NSLOT - 2) in flight, wait for all, scores of step 0
#pragma unroll
  for (int j = 0; j < NSLOT; ++j)
    if (j < total) {
      const uint32_t t = tile_at(j);
      stage_k(kbase + step_off(t, j), Ks[j]);
      if (j < NSLOT - 1) stage(a.v + step_off(t, j), Vs[j]);
    }
  asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
  f32x16 sc[KB / 32];
  scores(Ks[0], sc);
  hsap_lds_barrier();  // every wave has read K slot 0 before step 0 refills it
  const int32_t qstart = doc_window_start(a, docw, gq);
  const uint32_t span = (uint32_t)(gq - qstart);

  int sk = 0;  // s % NSLOT
  // Instruction order asked of the compiler for the block of a step (bf16 scores): four K-operand
  // reads ahead, then per score MFMA one LDS read and four vector instructions (the exponentials,
  // sums and conversions of this step), then per PV MFMA two V^T reads and three vector ones.
  auto block_order = []() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);  // LDS reads
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x406, 4, 0);  // VALU, SALU, transcendental
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x406, 3, 0);
    }
  };
  // one 64-key step: softmax and PV of step s from `sc`, scores of step s + 1 into `sn` (run twice
  // per loop iteration with the score arrays swapped; `par` is s % 2 as a compile-time constant:
  // with two slots every slot index is one)
  auto step = [&](int s, auto par, f32x16 (&sc)[KB / 32], f32x16 (&sn)[KB / 32]) __attribute__((always_inline)) {
    constexpr int PAR = decltype(par)::value;
    // the window of tile (s + NSLOT) / SUBS is needed now (rare vector load: every 64 tiles)
    if (s + NSLOT < total && ((s + NSLOT) / SUBS) >> 6 > win_hi) load_window(win_hi + 1);
    const uint32_t tile = tile_at(s);
    const float sl = FP8 ? fp8_step_scale(head_scale * kscale_s[chunk_of(tile)]) : head_scale;
    // s % NSLOT, (s + 1) % NSLOT and (s + NSLOT - 1) % NSLOT: this step's slot, the slot of the
    // next scores and of V's refill
    const int s0 = NSLOT == 2 ? PAR : sk;
    const int s1 = NSLOT == 2 ? PAR ^ 1 : (sk == NSLOT - 1 ? 0 : sk + 1);
    const int sv = NSLOT == 2 ? PAR ^ 1 : (sk == 0 ? NSLOT - 1 : sk - 1);
    const bool ldk = s + NSLOT < total, ldv = s + NSLOT - 1 < total;
    if (ldk) stage_k(kbase + step_off(tile_at(s + NSLOT), s + NSLOT), Ks[s0]);
    if (ldv) stage(a.v + step_off(tile_at(s + NSLOT - 1), s + NSLOT - 1), Vs[sv]);

    // Masked tile: a step whose keys no query of the wave may see is skipped (all its
    // probabilities would be 0: the running max, sum and O stay as they are), and one whose keys
    // every query of the wave may see needs no per-element mask.
    bool live = true;
    if (tile >> 31) {  // MASKED
      const int32_t r = (int32_t)global_pos(a.geom, chunk_of(tile), step_row0(tile, s)) - qstart;  // offset of key 0
      const bool none = r > (int32_t)span || r + (KB - 1) < 0;
      const bool all = r >= 0 && r + (KB - 1) <= (int32_t)span;
      live = __builtin_amdgcn_ballot_w64(!none) != 0;
      if (live && __builtin_amdgcn_ballot_w64(!all) != 0) {
        // key row of register j: r + 32 nb + c_row(j, hi), with the lane's 4 hi folded in once
        const int32_t rel0 = r + 4 * hi;
#pragma unroll
        for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if ((uint32_t)(rel0 + (32 * nb + c_row(j, 0))) > span) sc[nb][j] = NEG_INF;
      }
    }
    float m_use = 0.f;
    if (live) {
      float mx = sc[0][0];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sc[nb][j]);
      const float m_new = fmaxf(m_run, pair_max(mx) * sl);
      if (__builtin_amdgcn_ballot_w64(m_new > m_run + RESCALE_SLACK) != 0) {
        const float alpha = fast_exp2(m_run - (m_new == NEG_INF ? 0.f : m_new));
        l_run *= alpha;
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
        m_run = m_new;
      }
      m_use = m_run == NEG_INF ? 0.f : m_run;
    }

    if (live) {
      // the block: exponentials of this step (each 32-key half followed in the source by that
      // half's next-step score products, so nothing common is left to hoist above the branch),
      // then PV of this step
      __builtin_amdgcn_s_setprio(1);
      float rs = 0.f;
      bf16x8 pb[KB / 32][2];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float p = fast_exp2(__builtin_fmaf(sc[nb][j], sl, -m_use));
          rs += p;
          pb[nb][j >> 3][j & 7] = (__bf16)p;
        }
        if constexpr (FP8) {
          if (nb == 0) scores(Ks[s1], sn);
        } else {
          bf16x8 kf[D / 16];
#pragma unroll
          for (int kk = 0; kk < D / 16; ++kk) kf[kk] = *(const bf16x8*)(Ks[s1] + 32 * nb * D + rowoff[kk]);
          sn[nb] = f32x16{};
#pragma unroll
          for (int kk = 0; kk < D / 16; ++kk) sn[nb] = mfma32(kf[kk], qf[kk], sn[nb]);
        }
      }
      l_run += rs;

      const __bf16* V = Vs[s0];
#pragma unroll
      for (int nb = 0; nb < KB / 32; ++nb)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int rb = (32 * nb + 16 * half) * D;
#pragma unroll
          for (int mb = 0; mb < D / 32; ++mb) {
            const bf16x8 av = cat4(ds_read_tr16(V + rb + troff[mb][0]), ds_read_tr16(V + rb + 8 * D + troff[mb][1]));
            o[mb] = mfma32(av, pb[nb][half], o[mb]);
          }
        }
      if constexpr (!FP8) block_order();
      __builtin_amdgcn_s_setprio(0);
    } else {
      scores(Ks[s1], sn);
    }
    // K(s + 2) and V(s + 1) must have landed before the next step.  Three slots: they were
    // issued one step ago, and this step's own transfers (UK instructions for K, U for V) stay in
    // flight.  Two slots: they are this step's transfers.
    if constexpr (NSLOT == 3) {
      if (ldk && ldv) vm_wait_barrier<UK + U>();
      else if (ldk) vm_wait_barrier<UK>();
      else if (ldv) vm_wait_barrier<U>();
      else vm_wait_barrier<0>();
    } else {
      vm_wait_barrier<0>();
    }
    sk = s1;
  };
  f32x16 sn[KB / 32];
  for (int s = 0; s < total; s += 2) {
    step(s, std::integral_constant<int, 0>{}, sc, sn);
    if (s + 1 < total) step(s + 1, std::integral_constant<int, 1>{}, sn, sc);
  }

  l_run = pair_sum(l_run);
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  const float lse = l_run > 0.f ? (m_run + __log2f(l_run)) * 0.69314718055994530942f : NEG_INF;
  if (final_out) {
    __bf16* op = a.o_out + (qrow * a.hq + h) * D + 4 * hi;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const bf16x4 val{(__bf16)(o[mb][4 * grp] * inv), (__bf16)(o[mb][4 * grp + 1] * inv),
                         (__bf16)(o[mb][4 * grp + 2] * inv), (__bf16)(o[mb][4 * grp + 3] * inv)};
        *(bf16x4*)(op + 32 * mb + 8 * grp) = val;
      }
    if (hi == 0) a.lse_out[(int64_t)h * n + qrow] = lse;
  } else {
    float* op = a.o_part + (((int64_t)slot * n + qrow) * a.hq + h) * D + 4 * hi;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const f32x4 val{o[mb][4 * grp] * inv, o[mb][4 * grp + 1] * inv, o[mb][4 * grp + 2] * inv,
                        o[mb][4 * grp + 3] * inv};
        *(f32x4*)(op + 32 * mb + 8 * grp) = val;
      }
    if (hi == 0) a.lse_part[((int64_t)slot * a.hq + h) * n + qrow] = lse;
  }
}

template <int BN, int WAVES, bool FUSED, bool FP8 = false>
static hsap_status launch_dl(const FwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hq;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  if constexpr (!FUSED && !FP8) {
    if (!a.runs) {
      hipLaunchKernelGGL((attn_fwd_dl_kernel<BN, WAVES, false, false, true>), dim3((unsigned)blocks), dim3(64 * WAVES),
                         0, stream, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
      return HSAP_OK;
    }
  }
  hipLaunchKernelGGL((attn_fwd_dl_kernel<BN, WAVES, FUSED, FP8>), dim3((unsigned)blocks), dim3(64 * WAVES), 0, stream,
                     a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

template <int D, int BN, int WAVES, bool FUSED, bool FP8 = false>
static hsap_status launch(const FwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hq;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  if constexpr (!FUSED && !FP8) {
    if (!a.runs) {
      hipLaunchKernelGGL((attn_fwd_kernel<D, BN, WAVES, false, false, true>), dim3((unsigned)blocks), dim3(64 * WAVES),
                         0, stream, a);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
      return HSAP_OK;
    }
  }
  hipLaunchKernelGGL((attn_fwd_kernel<D, BN, WAVES, FUSED, FP8>), dim3((unsigned)blocks), dim3(64 * WAVES), 0, stream,
                     a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

// shared argument checks and dispatch of the partial and fused forwards (FP8: e4m3 Q and K)
template <bool FUSED, bool FP8 = false>
static hsap_status forward(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                           const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs, int64_t num_runs,
                           FwdArgs& a, hipStream_t s) {
  Geom geom;
  hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  if (num_runs < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_runs < 0");
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  if ((int64_t)desc->heads_kv * d * 64 > INT32_MAX) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "heads_kv too large");
  const bool shape_ok = (d == 128 || d == 64) && (bn == 128 || bn == 64) &&
                        (bm == 128 || bm == 64 || (bm == 256 && d == 128)) && (!FP8 || d == 128);
  if (FP8 && !shape_ok)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no fp8 forward kernel for head_dim=%d BM=%d BN=%d (head_dim 128; BM 64, 128 or 256; "
              "BN 64 or 128)", d, bm, bn);
  if (!shape_ok)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED,
              "no forward kernel for head_dim=%d BM=%d BN=%d (BM in {64, 128}, or 256 with d = 128; BN in {64, 128})",
              d, bm, bn);
  if (num_runs == 0) return HSAP_OK;
  if (!q || !k || !v || !(doc_start || a.cu) || (!runs && FUSED) || (runs && !tiles) || (!runs && a.num_tiles && !tiles))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v) & 15)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q, k and v must be 16-byte aligned");
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.doc_start = doc_start;
  a.tiles = tiles;
  a.runs = runs;
  a.geom = geom;
  a.shard = desc->shard.shard_id;
  a.hq = desc->heads_q;
  a.hkv = desc->heads_kv;
  a.group = desc->heads_q / desc->heads_kv;
  a.scale_log2 = desc->softmax_scale * 1.44269504088896340736f;
  // head_dim 128 with 128- or 256-row q-tiles: the direct-to-LDS kernel, whose packed tile
  // descriptors hold chunks below 256 and k-tiles below 2^23 (else the register-staged kernel)
  const bool dl = d == 128 && (bm == 128 || bm == 256) && geom.P <= kMaxDlChunks && geom.n / bn < kMaxDlKTiles;
  if constexpr (FP8) {
    if ((uintptr_t)q & 15 || (uintptr_t)k & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "fp8 q and k must be 16-byte aligned");
    if (dl && bm == 256)
      return bn == 128 ? launch_dl<128, 8, FUSED, true>(a, num_runs, s) : launch_dl<64, 8, FUSED, true>(a, num_runs, s);
    if (dl && bm == 128)
      return bn == 128 ? launch_dl<128, 4, FUSED, true>(a, num_runs, s) : launch_dl<64, 4, FUSED, true>(a, num_runs, s);
    const int w = bm / 32;
    if (bn == 128) return w == 2 ? launch<128, 128, 2, FUSED, true>(a, num_runs, s)
                        : w == 4 ? launch<128, 128, 4, FUSED, true>(a, num_runs, s)
                                 : launch<128, 128, 8, FUSED, true>(a, num_runs, s);
    return w == 2 ? launch<128, 64, 2, FUSED, true>(a, num_runs, s)
         : w == 4 ? launch<128, 64, 4, FUSED, true>(a, num_runs, s)
                  : launch<128, 64, 8, FUSED, true>(a, num_runs, s);
  } else {
#define HSAP_FWD_CASE(D_, BN_, W_) \
  if (d == D_ && bn == BN_ && bm == 32 * W_) return launch<D_, BN_, W_, FUSED>(a, num_runs, s);
  if (dl && bm == 256)
    return bn == 128 ? launch_dl<128, 8, FUSED>(a, num_runs, s) : launch_dl<64, 8, FUSED>(a, num_runs, s);
  if (dl && bm == 128)
    return bn == 128 ? launch_dl<128, 4, FUSED>(a, num_runs, s) : launch_dl<64, 4, FUSED>(a, num_runs, s);
  if (d == 128 && bm == 256)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "256-row q-tiles need sp_degree <= %d and fewer than 2^23 k-tiles per chunk",
              kMaxDlChunks);
  HSAP_FWD_CASE(128, 128, 4)
  HSAP_FWD_CASE(128, 64, 4)
  HSAP_FWD_CASE(128, 128, 2)
  HSAP_FWD_CASE(128, 64, 2)
  HSAP_FWD_CASE(64, 128, 4)
  HSAP_FWD_CASE(64, 64, 4)
  HSAP_FWD_CASE(64, 128, 2)
  HSAP_FWD_CASE(64, 64, 2)
#undef HSAP_FWD_CASE
  }
  HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no forward kernel for head_dim=%d BM=%d BN=%d", d, bm, bn);
}

// Workgroups of the bf16 partial forward resident on one compute unit, from the runtime's
// occupancy calculation for the kernel forward() dispatches for this shape (its registers, LDS
// and workgroup size); 0 when the shape has no kernel or the query fails.
template <typename Kernel>
static int blocks_per_cu(Kernel kernel, int threads) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, threads, 0) != hipSuccess) return 0;
  return blocks;
}

int fwd_resident_per_cu(const hsap_attn_desc* desc) {
  Geom geom;
  if (check_attn(desc, &geom) != HSAP_OK) return 0;
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  if (bn != 64 && bn != 128) return 0;
  const bool dl = d == 128 && (bm == 128 || bm == 256) && geom.P <= kMaxDlChunks && geom.n / bn < kMaxDlKTiles;
  if (dl && bm == 256)
    return bn == 128 ? blocks_per_cu(attn_fwd_dl_kernel<128, 8, false>, 512) : blocks_per_cu(attn_fwd_dl_kernel<64, 8, false>, 512);
  if (dl) return bn == 128 ? blocks_per_cu(attn_fwd_dl_kernel<128, 4, false>, 256) : blocks_per_cu(attn_fwd_dl_kernel<64, 4, false>, 256);
#define HSAP_OCC_CASE(D_, BN_, W_) \
  if (d == D_ && bn == BN_ && bm == 32 * W_) return blocks_per_cu(attn_fwd_kernel<D_, BN_, W_, false>, 64 * W_);
  HSAP_OCC_CASE(128, 128, 4)
  HSAP_OCC_CASE(128, 64, 4)
  HSAP_OCC_CASE(128, 128, 2)
  HSAP_OCC_CASE(128, 64, 2)
  HSAP_OCC_CASE(64, 128, 4)
  HSAP_OCC_CASE(64, 64, 4)
  HSAP_OCC_CASE(64, 128, 2)
  HSAP_OCC_CASE(64, 64, 2)
#undef HSAP_OCC_CASE
  return 0;
}

}  // namespace hsap

using namespace hsap;

extern "C" hsap_status hsap_fwd_resident_workgroups(const hsap_attn_desc* desc, int32_t* out) {
  clear_error();
  if (!out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "out is NULL");
  *out = 0;
  Geom geom;
  const hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "device query: %s", hipGetErrorString(e));
  const int per_cu = fwd_resident_per_cu(desc);
  if (per_cu <= 0)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no forward kernel occupancy for head_dim=%d BM=%d BN=%d", desc->head_dim,
              desc->shard.block_m, desc->shard.block_n);
  *out = per_cu * cus;
  return HSAP_OK;
}

extern "C" hsap_status hsap_partial_attn_fwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const int32_t* doc_start, const hsap_tile* tiles, int64_t num_tiles,
                                             float* o_part, float* lse_part, void* hip_stream) {
  clear_error();
  Geom geom;
  const hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  if (desc->chunk_id < 0 || desc->chunk_id >= geom.P)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "chunk_id %d outside [0, %d)", desc->chunk_id, geom.P);
  if (num_tiles < 0 || num_tiles > (int64_t(1) << 30)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad num_tiles %lld", (long long)num_tiles);
  if (!o_part || !lse_part || !doc_start) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_part & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_part must be 16-byte aligned");
  FwdArgs a{};
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.num_slots = 1;
  a.num_tiles = (int32_t)num_tiles;
  // one workgroup per (q-tile, head): each finds its q-tile's tiles in the list
  return forward<false>(desc, q, k, v, doc_start, tiles, nullptr, geom.n / desc->shard.block_m, a,
                        (hipStream_t)hip_stream);
}

extern "C" hsap_status hsap_partial_attn_fwd_runs(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                             int64_t num_runs, float* o_part, float* lse_part, int32_t num_slots,
                                             void* hip_stream) {
  clear_error();
  if (num_slots < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_slots < 1");
  if (num_runs > 0 && (!o_part || !lse_part)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_part & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_part must be 16-byte aligned");
  FwdArgs a{};
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.num_slots = num_slots;
  return forward<false>(desc, q, k, v, doc_start, tiles, runs, num_runs, a, (hipStream_t)hip_stream);
}

extern "C" hsap_status hsap_attn_fwd_fused(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                           const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                           int64_t num_runs, void* o_out, float* lse_out, void* hip_stream) {
  clear_error();
  if (num_runs > 0 && (!o_out || !lse_out)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_out & 7) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_out must be 8-byte aligned");
  FwdArgs a{};
  a.o_out = (__bf16*)o_out;
  a.lse_out = lse_out;
  a.num_slots = 1;
  return forward<true>(desc, q, k, v, doc_start, tiles, runs, num_runs, a, (hipStream_t)hip_stream);
}

extern "C" hsap_status hsap_partial_attn_fwd_fp8(const hsap_attn_desc* desc, const uint8_t* q8, const uint8_t* k8,
                                                 const void* v, const float* q_scale, const float* k_scale,
                                                 const int32_t* doc_start, const hsap_tile* tiles,
                                                 const hsap_run* runs, int64_t num_runs, float* o_part,
                                                 float* lse_part, int32_t num_slots, void* hip_stream) {
  clear_error();
  if (num_slots < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_slots < 1");
  if (num_runs > 0 && (!o_part || !lse_part || !q_scale || !k_scale))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_part & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_part must be 16-byte aligned");
  FwdArgs a{};
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.num_slots = num_slots;
  a.q_scale = q_scale;
  a.k_scale = k_scale;
  return forward<false, true>(desc, q8, k8, v, doc_start, tiles, runs, num_runs, a, (hipStream_t)hip_stream);
}

namespace hsap {

hsap_status executor_forward(const hsap_attn_desc* desc, bool fused, const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens, int32_t num_docs, const hsap_tile* tiles,
                             const hsap_run* runs, int64_t num_runs, float* o_part, float* lse_part,
                             int32_t num_slots, void* o_out, float* lse_out, hipStream_t stream) {
  if (!cu_seqlens || num_docs < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "no cumulative lengths");
  if (num_runs > 0 && (!o_out || !lse_out)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_out & 7) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_out must be 8-byte aligned");
  FwdArgs a{};
  a.o_out = (__bf16*)o_out;
  a.lse_out = lse_out;
  a.cu = cu_seqlens;
  a.num_docs = num_docs;
  if (fused) {
    a.num_slots = 1;
    return forward<true>(desc, q, k, v, nullptr, tiles, runs, num_runs, a, stream);
  }
  if (num_slots < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_slots < 1");
  if (num_runs > 0 && (!o_part || !lse_part)) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if ((uintptr_t)o_part & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_part must be 16-byte aligned");
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.num_slots = num_slots;
  return forward<false>(desc, q, k, v, nullptr, tiles, runs, num_runs, a, stream);
}

}  // namespace hsap
