// Partial attention forward: one shard's queries against the listed k-tiles of
// each K/V chunk ("computing" in the instruction table of the SAP section; the
// attention equation of the inter-group SP section under the packing mask).
//
// Work decomposition: one workgroup per (run, query head).  A run is one
// (chunk, q-tile) with its listed k-tiles.  The workgroup has WAVES waves;
// wave w owns 32 query rows, so BM = 32 * WAVES.
//
// Per k-tile: K rows are staged in LDS as [key][d] and V as its transpose
// [d][key]; the wave computes the scores transposed, S^T = K Q^T, with Q held
// in registers as the MFMA B operand.  In that orientation a lane holds one
// query (its column) and 16 keys per 32-key block, so the row max and row sum
// of the online softmax need only the lane itself and lane l ^ 32.  P (bf16)
// then feeds O^T += V^T P^T as the B operand straight from registers: the
// register order of the score block is the key order both MFMA operands use.
// Scores are scaled by softmax_scale * log2(e) so the exponentials are exp2.
// FULL tiles skip all mask arithmetic; MASKED tiles compare each key position
// with the query's document start and position.
#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

struct FwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const int32_t* doc_start;
  const hsap_tile* tiles;
  const hsap_run* runs;
  float* o_part;
  float* lse_part;
  Geom geom;
  int32_t shard;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  float scale_log2;
};

template <int D, int BN, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void attn_fwd_kernel(FwdArgs a) {
  constexpr int BM = 32 * WAVES;
  constexpr int NT = 64 * WAVES;
  constexpr int KS = D + 8;   // LDS row stride of K (bf16), padded against bank conflicts
  constexpr int VS = BN + 8;  // LDS row stride of V^T
  constexpr float NEG_INF = -__builtin_inff();
  __shared__ __attribute__((aligned(16))) __bf16 Ks[BN * KS];
  __shared__ __attribute__((aligned(16))) __bf16 Vt[D * VS];

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int run_idx = blockIdx.x / a.hq;
  const int h = blockIdx.x - run_idx * a.hq;
  const hsap_run run = a.runs[run_idx];
  const int c = run.chunk;
  const int g = h / a.group;
  const int64_t n = a.geom.n;

  const int64_t qrow = (int64_t)run.tile * BM + 32 * w + l32;  // shard-local query row of this lane
  const int64_t gq = global_pos(a.geom, a.shard, qrow);

  float m_run = NEG_INF, l_run = 0.f;
  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};

  if (run.count > 0) {
    bf16x8 qf[D / 16];
    const __bf16* qp = a.q + (qrow * a.hq + h) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) qf[kk] = *(const bf16x8*)(qp + 16 * kk);
    const int64_t qstart = a.doc_start[gq];
    const int64_t rstride = (int64_t)a.hkv * D;

    for (int it = 0; it < run.count; ++it) {
      const hsap_tile tile = a.tiles[run.first + it];
      const int64_t krow0 = (int64_t)tile.k_tile * BN;
      const int64_t gk0 = global_pos(a.geom, c, krow0);
      const int64_t off = (((int64_t)c * n + krow0) * a.hkv + g) * D;
      const __bf16* kb = a.k + off;
      const __bf16* vb = a.v + off;

      __syncthreads();  // the previous tile's LDS reads are done
#pragma unroll
      for (int i = tid; i < BN * D / 8; i += NT) {
        const int row = i / (D / 8), cc = i % (D / 8);
        const bf16x8 kv = *(const bf16x8*)(kb + row * rstride + cc * 8);
        const bf16x8 vv = *(const bf16x8*)(vb + row * rstride + cc * 8);
        *(bf16x8*)(Ks + row * KS + cc * 8) = kv;
#pragma unroll
        for (int e = 0; e < 8; ++e) Vt[(cc * 8 + e) * VS + row] = vv[e];
      }
      __syncthreads();

      // S^T = K Q^T, 32 keys per block
      f32x16 s[BN / 32];
#pragma unroll
      for (int nb = 0; nb < BN / 32; ++nb) {
        s[nb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk) {
          const bf16x8 af = *(const bf16x8*)(Ks + (32 * nb + l32) * KS + 16 * kk + 8 * hi);
          s[nb] = mfma32(af, qf[kk], s[nb]);
        }
      }
      if (tile.kind == HSAP_TILE_MASKED) {
#pragma unroll
        for (int nb = 0; nb < BN / 32; ++nb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int64_t gk = gk0 + 32 * nb + c_row(j, hi);
            if (gk < qstart || gk > gq) s[nb][j] = NEG_INF;
          }
      }
      // online softmax over this tile's keys (row = this lane's query)
      float mx = NEG_INF;
#pragma unroll
      for (int nb = 0; nb < BN / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[nb][j]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * a.scale_log2);
      const float m_use = m_new == NEG_INF ? 0.f : m_new;
      const float alpha = fast_exp2(m_run - m_use);
      float rs = 0.f;
#pragma unroll
      for (int nb = 0; nb < BN / 32; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float p = fast_exp2(s[nb][j] * a.scale_log2 - m_use);
          s[nb][j] = p;
          rs += p;
        }
      rs += __shfl_xor(rs, 32);
      l_run = l_run * alpha + rs;
      m_run = m_new;
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;

      // O^T += V^T P^T: 16 keys per MFMA
#pragma unroll
      for (int nb = 0; nb < BN / 32; ++nb)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          bf16x8 pb;
#pragma unroll
          for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[nb][8 * half + e];
#pragma unroll
          for (int mb = 0; mb < D / 32; ++mb) {
            const __bf16* vr = Vt + (32 * mb + l32) * VS + 32 * nb + 16 * half + 4 * hi;
            const bf16x8 av = cat4(*(const bf16x4*)vr, *(const bf16x4*)(vr + 8));
            o[mb] = mfma32(av, pb, o[mb]);
          }
        }
    }

    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    float* op = a.o_part + (((int64_t)c * n + qrow) * a.hq + h) * D + 4 * hi;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const f32x4 val{o[mb][4 * grp] * inv, o[mb][4 * grp + 1] * inv, o[mb][4 * grp + 2] * inv,
                        o[mb][4 * grp + 3] * inv};
        *(f32x4*)(op + 32 * mb + 8 * grp) = val;
      }
  }
  if (hi == 0)
    a.lse_part[((int64_t)c * a.hq + h) * n + qrow] =
        l_run > 0.f ? (m_run + __log2f(l_run)) * 0.69314718055994530942f : NEG_INF;
}

template <int D, int BN, int WAVES>
static hsap_status launch(const FwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hq;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  hipLaunchKernelGGL((attn_fwd_kernel<D, BN, WAVES>), dim3((unsigned)blocks), dim3(64 * WAVES), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_fwd launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

}  // namespace hsap

using namespace hsap;

extern "C" hsap_status hsap_partial_attn_fwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                             int64_t num_runs, float* o_part, float* lse_part, void* hip_stream) {
  clear_error();
  Geom geom;
  hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  if (num_runs < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_runs < 0");
  if (num_runs == 0) return HSAP_OK;
  if (!q || !k || !v || !doc_start || !tiles || !runs || !o_part || !lse_part)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o_part) & 15)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q, k, v and o_part must be 16-byte aligned");
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  FwdArgs a;
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.doc_start = doc_start;
  a.tiles = tiles;
  a.runs = runs;
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.geom = geom;
  a.shard = desc->shard.shard_id;
  a.hq = desc->heads_q;
  a.hkv = desc->heads_kv;
  a.group = desc->heads_q / desc->heads_kv;
  a.scale_log2 = desc->softmax_scale * 1.44269504088896340736f;
  hipStream_t s = (hipStream_t)hip_stream;
#define HSAP_FWD_CASE(D_, BN_, W_) \
  if (d == D_ && bn == BN_ && bm == 32 * W_) return launch<D_, BN_, W_>(a, num_runs, s);
  HSAP_FWD_CASE(128, 128, 4)
  HSAP_FWD_CASE(128, 64, 4)
  HSAP_FWD_CASE(128, 128, 2)
  HSAP_FWD_CASE(128, 64, 2)
  HSAP_FWD_CASE(64, 128, 4)
  HSAP_FWD_CASE(64, 64, 4)
  HSAP_FWD_CASE(64, 128, 2)
  HSAP_FWD_CASE(64, 64, 2)
#undef HSAP_FWD_CASE
  HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no forward kernel for head_dim=%d BM=%d BN=%d (BM, BN in {64, 128})", d, bm, bn);
}
