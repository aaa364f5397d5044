// Partial attention backward: gradients of one shard's attention with
// respect to its queries and to the listed k-tiles of each K/V chunk (the
// backward "computing" whose results the paper's per-rank code returns as dq
// and dkv messages, instruction table of the SAP section).
//
// Work decomposition: one workgroup per (run, K/V head).  A run is one
// (chunk, k-tile) with the q-tiles listed against it.  The workgroup has
// WAVES waves; wave w owns 32 keys (BN = 32 * WAVES) and keeps their K and V
// rows in registers and their dK, dV accumulators in registers for the whole
// run, looping over the query heads of its K/V head group and over the listed
// q-tiles in sub-tiles of 64 rows.  Per sub-tile:
//   S  = Q K^T and dP = dO V^T     (lane = key, registers = queries)
//   P  = exp2(S * scale*log2e - LSE*log2e) on allowed pairs, dS = P (dP - delta)
//   dV += P^T dO,  dK += dS^T Q     (A operands straight from registers)
//   dQ += scale * dS K              (dS through LDS; fp32 atomic adds)
// P is recomputed from the final (merged) LSE, so no attention matrix is
// stored between forward and backward.
#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

struct BwdArgs {
  const __bf16* q;
  const __bf16* k;
  const __bf16* v;
  const __bf16* d_o;
  const float* lse;
  const float* delta;
  const int32_t* doc_start;
  const hsap_tile* tiles;
  const hsap_run* runs;
  float* dq;
  float* dk;
  float* dv;
  Geom geom;
  int32_t shard;
  int32_t hq;
  int32_t hkv;
  int32_t group;
  int32_t bm;
  float scale;
  float scale_log2;
};

template <int D, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void attn_bwd_kernel(BwdArgs a) {
  constexpr int BN = 32 * WAVES;
  constexpr int NT = 64 * WAVES;
  constexpr int SUB = 64;      // query rows per LDS sub-tile
  constexpr int QS = D + 8;    // row stride of Qs / dOs  [query][d]
  constexpr int TS = SUB + 8;  // row stride of Qt / dOt  [d][query]
  constexpr int SS = BN + 8;   // row stride of dSs [query][key] and Kt [d][key]
  constexpr float LOG2E = 1.44269504088896340736f;
  __shared__ __attribute__((aligned(16))) __bf16 Qs[SUB * QS];
  __shared__ __attribute__((aligned(16))) __bf16 dOs[SUB * QS];
  __shared__ __attribute__((aligned(16))) __bf16 Qt[D * TS];
  __shared__ __attribute__((aligned(16))) __bf16 dOt[D * TS];
  __shared__ __attribute__((aligned(16))) __bf16 dSs[SUB * SS];
  __shared__ __attribute__((aligned(16))) __bf16 Kt[D * SS];
  __shared__ float lse_s[SUB];
  __shared__ float delta_s[SUB];
  __shared__ int32_t start_s[SUB];

  const int tid = threadIdx.x;
  const int w = tid >> 6, lane = tid & 63, l32 = lane & 31, hi = lane >> 5;
  const int run_idx = blockIdx.x / a.hkv;
  const int g = blockIdx.x - run_idx * a.hkv;
  const hsap_run run = a.runs[run_idx];
  const int c = run.chunk;
  const int64_t n = a.geom.n;
  const int64_t krow0 = (int64_t)run.tile * BN;
  const int64_t gk = global_pos(a.geom, c, krow0 + 32 * w + l32);  // this lane's key position
  const int64_t kvrow = (int64_t)c * n + krow0;                    // first row in the sharded K/V buffers

  // K and V rows of this lane's key as MFMA B operands; K^T of the whole tile in LDS
  bf16x8 kf[D / 16], vf[D / 16];
  {
    const int64_t off = ((kvrow + 32 * w + l32) * a.hkv + g) * D + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) {
      kf[kk] = *(const bf16x8*)(a.k + off + 16 * kk);
      vf[kk] = *(const bf16x8*)(a.v + off + 16 * kk);
    }
    for (int i = tid; i < BN * D / 8; i += NT) {
      const int row = i / (D / 8), cc = i % (D / 8);
      const bf16x8 x = *(const bf16x8*)(a.k + ((kvrow + row) * a.hkv + g) * D + cc * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) Kt[(cc * 8 + e) * SS + row] = x[e];
    }
  }

  f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) {
    dk[mb] = f32x16{};
    dv[mb] = f32x16{};
  }

  for (int hh = 0; hh < a.group; ++hh) {
    const int h = g * a.group + hh;
    for (int it = 0; it < run.count; ++it) {
      const hsap_tile tile = a.tiles[run.first + it];
      const bool masked = tile.kind == HSAP_TILE_MASKED;
      for (int sub = 0; sub < a.bm / SUB; ++sub) {
        const int64_t q0 = (int64_t)tile.q_tile * a.bm + sub * SUB;  // shard-local first row
        const int64_t gq0 = global_pos(a.geom, a.shard, q0);
        __syncthreads();  // previous sub-tile's LDS reads are done (and Kt is written)
        for (int i = tid; i < SUB * D / 8; i += NT) {
          const int row = i / (D / 8), cc = i % (D / 8);
          const int64_t src = ((q0 + row) * a.hq + h) * D + cc * 8;
          const bf16x8 x = *(const bf16x8*)(a.q + src);
          const bf16x8 y = *(const bf16x8*)(a.d_o + src);
          *(bf16x8*)(Qs + row * QS + cc * 8) = x;
          *(bf16x8*)(dOs + row * QS + cc * 8) = y;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            Qt[(cc * 8 + e) * TS + row] = x[e];
            dOt[(cc * 8 + e) * TS + row] = y[e];
          }
        }
        for (int i = tid; i < SUB; i += NT) {
          const float l = a.lse[(int64_t)h * n + q0 + i];
          lse_s[i] = l == -__builtin_inff() ? __builtin_inff() : l * LOG2E;  // a row with no key gets P = 0
          delta_s[i] = a.delta[(int64_t)h * n + q0 + i];
          start_s[i] = a.doc_start[gq0 + i];
        }
        __syncthreads();

        f32x16 p[SUB / 32], ds[SUB / 32];
#pragma unroll
        for (int qb = 0; qb < SUB / 32; ++qb) {
          f32x16 sacc{}, dpacc{};
#pragma unroll
          for (int kk = 0; kk < D / 16; ++kk) {
            const bf16x8 qa = *(const bf16x8*)(Qs + (32 * qb + l32) * QS + 16 * kk + 8 * hi);
            const bf16x8 da = *(const bf16x8*)(dOs + (32 * qb + l32) * QS + 16 * kk + 8 * hi);
            sacc = mfma32(qa, kf[kk], sacc);
            dpacc = mfma32(da, vf[kk], dpacc);
          }
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int qr = 32 * qb + c_row(j, hi);
            const bool ok = !masked || (start_s[qr] <= gk && gk <= gq0 + qr);
            const float pv = ok ? fast_exp2(sacc[j] * a.scale_log2 - lse_s[qr]) : 0.f;
            p[qb][j] = pv;
            ds[qb][j] = pv * (dpacc[j] - delta_s[qr]);
          }
        }
        // dV += P^T dO and dK += dS^T Q (16 queries per MFMA)
#pragma unroll
        for (int qb = 0; qb < SUB / 32; ++qb)
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            bf16x8 pa, sa;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              pa[e] = (__bf16)p[qb][8 * half + e];
              sa[e] = (__bf16)ds[qb][8 * half + e];
            }
#pragma unroll
            for (int mb = 0; mb < D / 32; ++mb) {
              const int o = (32 * mb + l32) * TS + 32 * qb + 16 * half + 4 * hi;
              dv[mb] = mfma32(pa, cat4(*(const bf16x4*)(dOt + o), *(const bf16x4*)(dOt + o + 8)), dv[mb]);
              dk[mb] = mfma32(sa, cat4(*(const bf16x4*)(Qt + o), *(const bf16x4*)(Qt + o + 8)), dk[mb]);
            }
          }
        // dS to LDS as [query][key] for the dQ product
#pragma unroll
        for (int qb = 0; qb < SUB / 32; ++qb)
#pragma unroll
          for (int j = 0; j < 16; ++j) dSs[(32 * qb + c_row(j, hi)) * SS + 32 * w + l32] = (__bf16)ds[qb][j];
        __syncthreads();
        // dQ[query, d] += scale * sum_key dS[query, key] K[key, d]; 32x32 blocks spread over the waves
        constexpr int NB = (SUB / 32) * (D / 32);
#pragma unroll
        for (int b = w; b < NB; b += WAVES) {
          const int qb = b / (D / 32), mb = b % (D / 32);
          f32x16 acc{};
#pragma unroll
          for (int ks = 0; ks < BN / 16; ++ks) {
            const bf16x8 sa = *(const bf16x8*)(dSs + (32 * qb + l32) * SS + 16 * ks + 8 * hi);
            const bf16x8 kb = *(const bf16x8*)(Kt + (32 * mb + l32) * SS + 16 * ks + 8 * hi);
            acc = mfma32(sa, kb, acc);
          }
          float* dst = a.dq + ((q0 + 32 * qb) * a.hq + h) * D + 32 * mb + l32;
#pragma unroll
          for (int j = 0; j < 16; ++j) unsafeAtomicAdd(dst + (int64_t)c_row(j, hi) * a.hq * D, acc[j] * a.scale);
        }
      }
    }
  }

  // this workgroup owns rows [krow0, krow0 + BN) of chunk c for K/V head g: plain read-add-write
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int64_t idx = ((kvrow + 32 * w + c_row(j, hi)) * a.hkv + g) * D + 32 * mb + l32;
      a.dk[idx] += dk[mb][j] * a.scale;
      a.dv[idx] += dv[mb][j];
    }
}

template <int D, int WAVES>
static hsap_status launch_bwd(const BwdArgs& a, int64_t num_runs, hipStream_t stream) {
  const int64_t blocks = num_runs * a.hkv;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many runs x heads");
  hipLaunchKernelGGL((attn_bwd_kernel<D, WAVES>), dim3((unsigned)blocks), dim3(64 * WAVES), 0, stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "attn_bwd launch: %s", hipGetErrorString(e));
  return HSAP_OK;
}

}  // namespace hsap

using namespace hsap;

extern "C" hsap_status hsap_partial_attn_bwd(const hsap_attn_desc* desc, const void* q, const void* k, const void* v,
                                             const void* d_o, const float* lse, const float* delta,
                                             const int32_t* doc_start, const hsap_tile* tiles, const hsap_run* runs,
                                             int64_t num_runs, float* dq_acc, float* dk_acc, float* dv_acc,
                                             void* hip_stream) {
  clear_error();
  Geom geom;
  hsap_status st = check_attn(desc, &geom);
  if (st != HSAP_OK) return st;
  if (num_runs < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_runs < 0");
  if (num_runs == 0) return HSAP_OK;
  if (!q || !k || !v || !d_o || !lse || !delta || !doc_start || !tiles || !runs || !dq_acc || !dk_acc || !dv_acc)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)d_o) & 15)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q, k, v and d_o must be 16-byte aligned");
  const int bm = desc->shard.block_m, bn = desc->shard.block_n, d = desc->head_dim;
  if (bm % 64) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "backward needs BM a multiple of 64 (BM=%d)", bm);
  BwdArgs a;
  a.q = (const __bf16*)q;
  a.k = (const __bf16*)k;
  a.v = (const __bf16*)v;
  a.d_o = (const __bf16*)d_o;
  a.lse = lse;
  a.delta = delta;
  a.doc_start = doc_start;
  a.tiles = tiles;
  a.runs = runs;
  a.dq = dq_acc;
  a.dk = dk_acc;
  a.dv = dv_acc;
  a.geom = geom;
  a.shard = desc->shard.shard_id;
  a.hq = desc->heads_q;
  a.hkv = desc->heads_kv;
  a.group = desc->heads_q / desc->heads_kv;
  a.bm = bm;
  a.scale = desc->softmax_scale;
  a.scale_log2 = desc->softmax_scale * 1.44269504088896340736f;
  hipStream_t s = (hipStream_t)hip_stream;
  if (d == 128 && bn == 128) return launch_bwd<128, 4>(a, num_runs, s);
  if (d == 128 && bn == 64) return launch_bwd<128, 2>(a, num_runs, s);
  if (d == 64 && bn == 64) return launch_bwd<64, 2>(a, num_runs, s);
  HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "no backward kernel for head_dim=%d BN=%d", d, bn);
}
