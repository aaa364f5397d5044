// Memory-bound kernels of libhsap: the LSE merge of partial results, the
// backward's row term delta = rowsum(dO * O), fp32 -> bf16 conversion, the
// per-position document start, the gather into sharded order, and the e4m3
// quantisation of Q and K for the fp8 score variant.
#include <algorithm>
#include <mutex>

#include "hsap_internal.h"
#include "mfma.h"

namespace hsap {

// ---------------------------------------------------------------------------
// LSE merge (online-softmax combination of the ring's partial results)
//
// Work unit: one wave merges one head's 16 consecutive rows, so the LSE values
// it reads and writes per part are one 64-byte line, and each O row (D fp32
// per part) is read by D/4 lanes, 16 bytes each.  Parts whose LSE is -inf
// are never read.
// ---------------------------------------------------------------------------
struct MergeArgs {
  const float* o[HSAP_MAX_MERGE_PARTS];
  const float* lse[HSAP_MAX_MERGE_PARTS];
  int32_t num_parts;
  int32_t hq;
  int64_t n;
  __bf16* o_out;
  float* lse_out;
  // Rows to merge: with `tiles` NULL every row 0..n-1; otherwise the BM-row q-tiles listed in
  // tiles[0 .. num_tiles-1], as "merge rows" v = 0 .. num_tiles * BM - 1 standing for shard row
  // tiles[v / BM] * BM + v % BM (the other q-tiles' rows are already final: not read, not written).
  const int32_t* tiles;
  int64_t rows;  // merge rows: n, or num_tiles * BM
  int32_t bm;
};

// shard row of merge row v
__device__ __forceinline__ int64_t merge_row(const MergeArgs& a, int64_t v) {
  if (!a.tiles) return v;
  const int64_t t = v / a.bm;
  return (int64_t)a.tiles[t] * a.bm + (v - t * a.bm);
}

// Few parts (num_parts <= PR): one wave merges one head's 16 consecutive rows.
// Lane i reads (and finally writes) the LSE of row i & 15, so each part's LSE
// values for the group are one 64-byte line; the per-row weights then move to
// the lanes that handle the O rows (2 rows of D fp32 per wave instruction, D/4
// lanes per row) with a lane permute.  Each instruction's loads for every part
// are issued together; few registers per wave keep many waves resident, which
// is what keeps the loads in flight (holding a whole group's loads per wave
// measured slower).
template <int D, int PR>
__global__ __launch_bounds__(256) void lse_merge_few_kernel(MergeArgs a) {
  constexpr int RPI = 256 / D;              // rows per wave instruction: 64 lanes x 4 floats / D
  constexpr int STEPS = 16 / RPI;           // instructions per 16-row group
  constexpr float NEG_INF = -__builtin_inff();
  constexpr float LOG2E = 1.44269504088896340736f;
  constexpr float LN2 = 0.69314718055994530942f;
  const int lane = threadIdx.x & 63;
  const int64_t groups_per_head = (a.rows + 15) / 16;
  const int64_t groups = groups_per_head * a.hq;
  const int64_t wave0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) / 64;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int sub = lane / (D / 4);           // which row of an instruction this lane serves
  const int d0 = 4 * (lane % (D / 4));      // its 4 consecutive d
  for (int64_t grp = wave0; grp < groups; grp += waves) {
    const int64_t h = grp / groups_per_head;
    const int64_t v0 = (grp - h * groups_per_head) * 16;
    // a 16-row group never straddles listed q-tiles (BM % 16 == 0): its shard rows are r0 + 0..15
    const int64_t r0 = merge_row(a, v0);
    // LSE of row r0 + (lane & 15) for every part; max and result in natural-log units, only
    // differences scaled to log2 units, so a row with one finite part keeps its LSE exactly
    const int64_t my_row = r0 + (lane & 15);
    const bool row_ok = v0 + (lane & 15) < a.rows;
    float l[PR];
#pragma unroll
    for (int p = 0; p < PR; ++p) l[p] = (p < a.num_parts && row_ok) ? a.lse[p][h * a.n + my_row] : NEG_INF;
    float mx = l[0];
#pragma unroll
    for (int p = 1; p < PR; ++p) mx = fmaxf(mx, l[p]);
    float sum = 0.f;
#pragma unroll
    for (int p = 0; p < PR; ++p) sum += l[p] == NEG_INF ? 0.f : fast_exp2((l[p] - mx) * LOG2E);
    const float Lm = mx == NEG_INF ? NEG_INF : mx + __log2f(sum) * LN2;
    float wl[PR];
#pragma unroll
    for (int p = 0; p < PR; ++p) wl[p] = l[p] == NEG_INF ? 0.f : fast_exp2((l[p] - Lm) * LOG2E);
    // O rows: instruction k covers rows r0 + RPI * k + sub
#pragma unroll
    for (int k = 0; k < STEPS; ++k) {
      const int j = RPI * k + sub;  // row within the group; its weights live in lane j
      const int64_t row = r0 + j;
      const bool in = v0 + j < a.rows;
      float w[PR];
      f32x4 x[PR];
#pragma unroll
      for (int p = 0; p < PR; ++p) {
        w[p] = __int_as_float(__builtin_amdgcn_ds_bpermute(4 * j, __float_as_int(wl[p])));
        x[p] = (w[p] > 0.f && in) ? *(const f32x4*)(a.o[p] + (row * a.hq + h) * D + d0)
                                  : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      if (!in) continue;
      f32x4 acc{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < PR; ++p) acc += w[p] * x[p];
      const bf16x4 out{(__bf16)acc[0], (__bf16)acc[1], (__bf16)acc[2], (__bf16)acc[3]};
      *(bf16x4*)(a.o_out + (row * a.hq + h) * D + d0) = out;
    }
    if (lane < 16 && row_ok) a.lse_out[h * a.n + my_row] = Lm;
  }
}

// Many parts (up to HSAP_MAX_MERGE_PARTS): one wave per (head, 16-row group) as in the
// few-parts kernel, with lane = row + 16 g reading the LSEs of parts g, g + 4, g + 8, ... of its
// row, so each lane holds at most a quarter of them.  Max and sum are combined over the four
// lanes of a row with lane permutes (max and result in natural-log units, differences scaled to
// log2 units, as in the few-parts kernel: a single finite part passes through exactly); the
// weights go to LDS, and the O pass then walks the parts with no LSE load in front of any O load
// (issuing the next part's loads before accumulating the current one measured slower: more
// registers, fewer resident waves).
template <int D>
__global__ __launch_bounds__(256) void lse_merge_many_kernel(MergeArgs a) {
  constexpr int RPI = 256 / D;                       // rows per wave instruction
  constexpr int STEPS = 16 / RPI;                    // instructions per 16-row group
  constexpr int LPER = HSAP_MAX_MERGE_PARTS / 4;     // parts per lane
  constexpr float NEG_INF = -__builtin_inff();
  constexpr float LOG2E = 1.44269504088896340736f;
  constexpr float LN2 = 0.69314718055994530942f;
  __shared__ float w_s[4][HSAP_MAX_MERGE_PARTS][16];  // per wave: weight of (part, row of the group)
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int r16 = lane & 15, pg = lane >> 4;
  const int sub = lane / (D / 4);                    // row of an instruction this lane serves
  const int d0 = 4 * (lane % (D / 4));
  const int np = a.num_parts;
  const int64_t groups_per_head = (a.rows + 15) / 16;
  const int64_t groups = groups_per_head * a.hq;
  const int64_t waves = (int64_t)gridDim.x * 4;
  for (int64_t grp = (int64_t)blockIdx.x * 4 + wv; grp < groups; grp += waves) {
    const int64_t h = grp / groups_per_head;
    const int64_t v0 = (grp - h * groups_per_head) * 16;
    const int64_t r0 = merge_row(a, v0);  // the group's shard rows are r0 + 0..15 (BM % 16 == 0)
    const bool row_ok = v0 + r16 < a.rows;
    float l[LPER];
    float mx = NEG_INF;
#pragma unroll
    for (int j = 0; j < LPER; ++j) {
      const int p = pg + 4 * j;
      l[j] = (p < np && row_ok) ? a.lse[p][h * a.n + r0 + r16] : NEG_INF;
      mx = fmaxf(mx, l[j]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < LPER; ++j) sum += l[j] == NEG_INF ? 0.f : fast_exp2((l[j] - mx) * LOG2E);
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    const float Lm = mx == NEG_INF ? NEG_INF : mx + __log2f(sum) * LN2;
#pragma unroll
    for (int j = 0; j < LPER; ++j) {
      const int p = pg + 4 * j;
      if (p < np) w_s[wv][p][r16] = l[j] == NEG_INF ? 0.f : fast_exp2((l[j] - Lm) * LOG2E);
    }
    __builtin_amdgcn_wave_barrier();  // a wave's LDS accesses complete in order: the weights are there
    // O pass: instruction k covers rows RPI k + sub of the group
    f32x4 acc[STEPS], x[STEPS];
    float wk[STEPS];
    auto load = [&](int p, f32x4 (&xs)[STEPS], float (&ws)[STEPS]) {
#pragma unroll
      for (int k = 0; k < STEPS; ++k) {
        const int j = RPI * k + sub;
        ws[k] = w_s[wv][p][j];
        xs[k] = (ws[k] > 0.f && v0 + j < a.rows) ? *(const f32x4*)(a.o[p] + ((r0 + j) * a.hq + h) * D + d0)
                                                 : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };
#pragma unroll
    for (int k = 0; k < STEPS; ++k) acc[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int p = 0; p < np; ++p) {
      load(p, x, wk);
#pragma unroll
      for (int k = 0; k < STEPS; ++k) acc[k] += wk[k] * x[k];
    }
#pragma unroll
    for (int k = 0; k < STEPS; ++k) {
      const int j = RPI * k + sub;
      if (v0 + j >= a.rows) continue;
      const bf16x4 out{(__bf16)acc[k][0], (__bf16)acc[k][1], (__bf16)acc[k][2], (__bf16)acc[k][3]};
      *(bf16x4*)(a.o_out + ((r0 + j) * a.hq + h) * D + d0) = out;
    }
    if (pg == 0 && row_ok) a.lse_out[h * a.n + r0 + r16] = Lm;
    __builtin_amdgcn_wave_barrier();  // the next group's weights overwrite w_s only after every read
  }
}

// ---------------------------------------------------------------------------
// delta[h, i] = sum_d dO[i, h, d] * O[i, h, d]
// D/8 lanes per (row, head), 8 bf16 each, reduced with lane shuffles.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_preprocess_kernel(const __bf16* o, const __bf16* d_o, int64_t n, int32_t hq,
                                                             float* delta) {
  constexpr int TPR = D / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t rh = gid / TPR;
  const int part = (int)(gid % TPR);
  const bool live = rh < n * hq;
  float acc = 0.f;
  if (live) {
    const bf16x8 x = *(const bf16x8*)(o + rh * D + 8 * part);
    const bf16x8 y = *(const bf16x8*)(d_o + rh * D + 8 * part);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = __builtin_fmaf((float)x[e], (float)y[e], acc);
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (live && part == 0) {
    const int64_t row = rh / hq;
    const int h = (int)(rh - row * hq);
    delta[(int64_t)h * n + row] = acc;
  }
}

// ---------------------------------------------------------------------------
// fp32 -> bf16 (round to nearest even), 8 elements per thread when aligned
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void convert_kernel(const float* src, __bf16* dst, int64_t count, int vec) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i * 8 < count; i += stride) {
    if (vec && i * 8 + 8 <= count) {
      const f32x4 a = *(const f32x4*)(src + i * 8);
      const f32x4 b = *(const f32x4*)(src + i * 8 + 4);
      const bf16x8 out{(__bf16)a[0], (__bf16)a[1], (__bf16)a[2], (__bf16)a[3],
                       (__bf16)b[0], (__bf16)b[1], (__bf16)b[2], (__bf16)b[3]};
      *(bf16x8*)(dst + i * 8) = out;
    } else {
      for (int64_t j = i * 8; j < i * 8 + 8 && j < count; ++j) dst[j] = (__bf16)src[j];
    }
  }
}

// ---------------------------------------------------------------------------
// doc_start[t] = cu[k] for the last k with cu[k] <= t (binary search)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void doc_start_kernel(const int32_t* cu, int32_t num_docs, int64_t total,
                                                        int32_t* out) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += stride) {
    int32_t lo = 0, hi = num_docs;  // invariant: cu[lo] <= t < cu[hi]
    while (hi - lo > 1) {
      const int32_t mid = (lo + hi) >> 1;
      if (cu[mid] <= t) lo = mid;
      else hi = mid;
    }
    out[t] = cu[lo];
  }
}

// ---------------------------------------------------------------------------
// dst[c, l] = src[position of chunk c's local row l], 16 bytes per lane
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_kernel(Geom g, const uint4* src, uint4* dst, int64_t words_per_row) {
  const int64_t total = g.N * words_per_row;
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += stride) {
    const int64_t row = i / words_per_row, word = i - row * words_per_row;
    const int32_t c = (int32_t)(row / g.n);
    const int64_t local = row - (int64_t)c * g.n;
    dst[i] = src[global_pos(g, c, local) * words_per_row + word];
  }
}

// ---------------------------------------------------------------------------
// zero fill, 16 bytes per lane (a kernel rather than a memset node, so the
// sequence stays valid inside captured graphs)
// ---------------------------------------------------------------------------
// Zeroes the listed tiles of two buffers: entry i names tile list[i], the byte range
// [list[i] * tile_words * 16, +tile_words * 16) of both a and b.  blockIdx.x is the entry.
__global__ __launch_bounds__(256) void zero_tiles_kernel(uint4* a, uint4* b, const int32_t* list, int64_t tile_words) {
  const int64_t base = (int64_t)list[blockIdx.x] * tile_words;
  for (int64_t i = (int64_t)blockIdx.y * 256 + threadIdx.x; i < tile_words; i += (int64_t)gridDim.y * 256) {
    a[base + i] = uint4{0, 0, 0, 0};
    b[base + i] = uint4{0, 0, 0, 0};
  }
}

// ---------------------------------------------------------------------------
// e4m3 quantisation of x [G, rows, H, d]: each (group g, head h) slice is cut
// into QSPLIT row ranges.  Pass 1: one workgroup per range writes the range's
// amax to the workspace.  Pass 2: one workgroup per range takes the slice's
// amax from its QSPLIT partial maxima, writes scale = amax / 448 (range 0),
// and converts its rows: code = e4m3(clamp(x * 448 / amax, +-448)) with the
// hardware's round-to-nearest-even conversion (which without the clamp would
// turn values beyond 448 into NaN codes).
// ---------------------------------------------------------------------------
constexpr int QSPLIT = HSAP_QUANT_SPLIT;

struct QuantArgs {
  const __bf16* x;
  int64_t rows;
  int32_t heads, d;
  uint8_t* out;
  float* scale;
  float* partial;  // [G * H * QSPLIT]
};

// the 16-byte chunks [c0, c1) of slice gh's row range s, and the element offset of chunk i
struct QuantRange {
  int64_t c0, c1, g;
  int32_t h, per_row;
  __device__ QuantRange(const QuantArgs& a, int gh, int s) {
    g = gh / a.heads;
    h = gh - (int32_t)g * a.heads;
    per_row = a.d / 8;
    const int64_t r0 = a.rows * s / QSPLIT, r1 = a.rows * (s + 1) / QSPLIT;
    c0 = r0 * per_row;
    c1 = r1 * per_row;
  }
  __device__ int64_t offset(const QuantArgs& a, int64_t i) const {
    const int64_t r = i / per_row;
    return ((g * a.rows + r) * a.heads + h) * a.d + (i - r * per_row) * 8;
  }
};

__device__ inline float block_max_256(float v, float* part) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));
}

__global__ __launch_bounds__(256) void quantize_amax_kernel(QuantArgs a) {
  __shared__ float part[4];
  const int gh = blockIdx.x / QSPLIT, sp = blockIdx.x - gh * QSPLIT;
  const QuantRange q(a, gh, sp);
  float amax = 0.f;
  for (int64_t i = q.c0 + threadIdx.x; i < q.c1; i += 256) {
    const bf16x8 v = *(const bf16x8*)(a.x + q.offset(a, i));
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)v[e]));
  }
  amax = block_max_256(amax, part);
  if (threadIdx.x == 0) a.partial[blockIdx.x] = amax;
}

__global__ __launch_bounds__(256) void quantize_convert_kernel(QuantArgs a) {
  const int gh = blockIdx.x / QSPLIT, sp = blockIdx.x - gh * QSPLIT;
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < QSPLIT; ++i) amax = fmaxf(amax, a.partial[gh * QSPLIT + i]);
  const float inv = amax > 0.f ? 448.f / amax : 0.f;
  if (sp == 0 && threadIdx.x == 0) a.scale[gh] = amax > 0.f ? amax / 448.f : 0.f;
  const QuantRange q(a, gh, sp);
  for (int64_t i = q.c0 + threadIdx.x; i < q.c1; i += 256) {
    const int64_t o = q.offset(a, i);
    const bf16x8 v = *(const bf16x8*)(a.x + o);
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = fminf(fmaxf((float)v[e] * inv, -448.f), 448.f);
    int lo = 0, hi = 0;
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], lo, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], lo, true);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(y[4], y[5], hi, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(y[6], y[7], hi, true);
    *(uint2*)(a.out + o) = make_uint2((uint32_t)lo, (uint32_t)hi);
  }
}

static hsap_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "%s launch: %s", what, hipGetErrorString(e));
  return HSAP_OK;
}

static unsigned grid_for(int64_t threads) {
  const int64_t b = (threads + 255) / 256;
  return (unsigned)(b < 1 ? 1 : (b > 65536 ? 65536 : b));
}

hsap_status zero_tiles(void* a, void* b, const int32_t* tiles, int32_t num_tiles, int64_t tile_bytes,
                       hipStream_t stream) {
  if (num_tiles == 0) return HSAP_OK;
  if (!a || !b || !tiles || num_tiles < 0 || tile_bytes <= 0 || (tile_bytes & 15) || (((uintptr_t)a | (uintptr_t)b) & 15))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "zero_tiles: bad buffers, list or tile size %lld", (long long)tile_bytes);
  const int64_t words = tile_bytes / 16;
  const unsigned per_tile = (unsigned)std::min<int64_t>(64, (words + 1023) / 1024);  // about 4 stores per thread
  hipLaunchKernelGGL(zero_tiles_kernel, dim3((unsigned)num_tiles, per_tile), dim3(256), 0, stream, (uint4*)a,
                     (uint4*)b, tiles, words);
  return check_launch("zero_tiles");
}

}  // namespace hsap

using namespace hsap;

extern "C" {

hsap_status hsap_lse_merge(int32_t num_parts, const float* const* o_parts, const float* const* lse_parts, int64_t n,
                           int32_t heads_q, int32_t head_dim, void* o_out, float* lse_out, void* hip_stream) {
  clear_error();
  return lse_merge(num_parts, o_parts, lse_parts, n, heads_q, head_dim, o_out, lse_out, nullptr, 0, 1,
                   (hipStream_t)hip_stream);
}

}  // extern "C"

namespace hsap {

hsap_status lse_merge(int32_t num_parts, const float* const* o_parts, const float* const* lse_parts, int64_t n,
                      int32_t heads_q, int32_t head_dim, void* o_out, float* lse_out, const int32_t* tiles,
                      int32_t num_tiles, int32_t block_m, hipStream_t s) {
  if (num_parts < 1 || num_parts > HSAP_MAX_MERGE_PARTS)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_parts %d outside 1..%d", num_parts, HSAP_MAX_MERGE_PARTS);
  if (!o_parts || !lse_parts || !o_out || !lse_out) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (n < 0 || heads_q <= 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad n=%lld or heads_q=%d", (long long)n, heads_q);
  if (head_dim != 64 && head_dim != 128) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "head_dim %d not supported", head_dim);
  MergeArgs a;
  for (int p = 0; p < num_parts; ++p) {
    if (!o_parts[p] || !lse_parts[p]) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "part %d pointer is NULL", p);
    if ((uintptr_t)o_parts[p] & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_parts[%d] not 16-byte aligned", p);
    a.o[p] = o_parts[p];
    a.lse[p] = lse_parts[p];
  }
  if ((uintptr_t)o_out & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o_out not 16-byte aligned");
  if (n == 0) return HSAP_OK;
  a.num_parts = num_parts;
  a.hq = heads_q;
  a.n = n;
  a.o_out = (__bf16*)o_out;
  a.lse_out = lse_out;
  if (tiles && (block_m < 16 || block_m % 16 || num_tiles < 0 || (int64_t)num_tiles * block_m > n))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "q-tile list needs BM a multiple of 16 and at most n / BM tiles");
  a.tiles = tiles;
  a.bm = tiles ? block_m : 1;
  a.rows = tiles ? (int64_t)num_tiles * block_m : n;
  if (a.rows == 0) return HSAP_OK;
  const dim3 block(256);
  if (num_parts <= 4) {
    // one wave per (head, 16 rows) group, four waves per block, grid-stride beyond 65536 blocks
    const int64_t groups = ((a.rows + 15) / 16) * heads_q;
    const dim3 grid((unsigned)std::min<int64_t>((groups + 3) / 4, 65536));
    if (head_dim == 128) {
      if (num_parts <= 2) hipLaunchKernelGGL((lse_merge_few_kernel<128, 2>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((lse_merge_few_kernel<128, 4>), grid, block, 0, s, a);
    } else {
      if (num_parts <= 2) hipLaunchKernelGGL((lse_merge_few_kernel<64, 2>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((lse_merge_few_kernel<64, 4>), grid, block, 0, s, a);
    }
  } else {
    const int64_t groups = ((a.rows + 15) / 16) * heads_q;
    const dim3 grid((unsigned)std::min<int64_t>((groups + 3) / 4, 65536));
    if (head_dim == 128) hipLaunchKernelGGL((lse_merge_many_kernel<128>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((lse_merge_many_kernel<64>), grid, block, 0, s, a);
  }
  return check_launch("lse_merge");
}

}  // namespace hsap

extern "C" {

hsap_status hsap_attn_bwd_preprocess(const void* o, const void* d_o, int64_t n, int32_t heads_q, int32_t head_dim,
                                     float* delta, void* hip_stream) {
  clear_error();
  if (!o || !d_o || !delta) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (n < 0 || heads_q <= 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad n=%lld or heads_q=%d", (long long)n, heads_q);
  if (head_dim != 64 && head_dim != 128) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "head_dim %d not supported", head_dim);
  if (((uintptr_t)o | (uintptr_t)d_o) & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "o and d_o must be 16-byte aligned");
  if (n == 0) return HSAP_OK;
  const int64_t threads = n * heads_q * (head_dim / 8);
  const int64_t blocks = (threads + 255) / 256;
  if (blocks > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "problem too large");
  hipStream_t s = (hipStream_t)hip_stream;
  if (head_dim == 128)
    hipLaunchKernelGGL(bwd_preprocess_kernel<128>, dim3((unsigned)blocks), dim3(256), 0, s, (const __bf16*)o,
                       (const __bf16*)d_o, n, heads_q, delta);
  else
    hipLaunchKernelGGL(bwd_preprocess_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, s, (const __bf16*)o,
                       (const __bf16*)d_o, n, heads_q, delta);
  return check_launch("bwd_preprocess");
}

hsap_status hsap_convert_f32_bf16(const float* src, void* dst, int64_t count, void* hip_stream) {
  clear_error();
  if (count < 0) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "count < 0");
  if (count == 0) return HSAP_OK;
  if (!src || !dst) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  const int vec = (((uintptr_t)src | (uintptr_t)dst) & 15) == 0;
  hipLaunchKernelGGL(convert_kernel, dim3(grid_for((count + 7) / 8)), dim3(256), 0, (hipStream_t)hip_stream, src,
                     (__bf16*)dst, count, vec);
  return check_launch("convert");
}

}  // extern "C"

namespace hsap {

// Shape and pointer checks of both quantisation entry points (the workspace is checked apart).
static hsap_status check_quantize(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                                  const uint8_t* codes, const float* scale) {
  if (groups < 1 || rows < 1 || heads < 1 || head_dim < 8 || head_dim % 8)
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad shape: groups %d, rows %lld, heads %d, head_dim %d (a multiple of 8)", groups,
              (long long)rows, heads, head_dim);
  if ((int64_t)groups * heads * QSPLIT > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "too many groups x heads");
  if (!x || !codes || !scale) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (((uintptr_t)x & 15) || ((uintptr_t)codes & 7))
    HSAP_FAIL(HSAP_ERR_INVALID_ARG, "x must be 16-byte and codes 8-byte aligned");
  return HSAP_OK;
}

// The two launches of the quantisation: per-range maxima into `workspace` (every entry written),
// then the slice maxima, scales and codes.
static hsap_status quantize(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                            uint8_t* codes, float* scale, float* workspace, hipStream_t stream) {
  const QuantArgs a{(const __bf16*)x, rows, heads, head_dim, codes, scale, workspace};
  const dim3 grid((unsigned)(groups * heads * QSPLIT));
  hipLaunchKernelGGL(quantize_amax_kernel, grid, dim3(256), 0, stream, a);
  hsap_status st = check_launch("quantize_fp8 amax");
  if (st != HSAP_OK) return st;
  hipLaunchKernelGGL(quantize_convert_kernel, grid, dim3(256), 0, stream, a);
  return check_launch("quantize_fp8 convert");
}

// Scratch of hsap_quantize_fp8_noalloc: the per-range maxima of up to
// HSAP_QUANT_NOALLOC_MAX_SLICES (group, head) slices.  Every device the library runs on holds its
// own copy (512 KiB) until the process ends.  Host code never uses this name as an address: each
// device's copy is reached through the address hipGetSymbolAddress returns for it.
static __device__ __align__(256) float scratch[HSAP_QUANT_NOALLOC_MAX_SLICES * QSPLIT];

constexpr int kMaxScratchDevices = 64;
static std::mutex scratch_mutex;
static float* scratch_addr[kMaxScratchDevices];  // per device, resolved on the first call there

// The device address of the current device's `scratch`, looked up once per device with that
// device current.
static hsap_status scratch_for_current_device(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) HSAP_FAIL(HSAP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices) HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      HSAP_FAIL(HSAP_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    scratch_addr[dev] = (float*)p;
  }
  *out = scratch_addr[dev];
  return HSAP_OK;
}

}  // namespace hsap

extern "C" {

hsap_status hsap_quantize_fp8(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                              uint8_t* codes, float* scale, float* workspace, void* hip_stream) {
  clear_error();
  const hsap_status st = check_quantize(x, groups, rows, heads, head_dim, codes, scale);
  if (st != HSAP_OK) return st;
  if (!workspace) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL workspace");
  return quantize(x, groups, rows, heads, head_dim, codes, scale, workspace, (hipStream_t)hip_stream);
}

hsap_status hsap_quantize_fp8_noalloc(const void* x, int32_t groups, int64_t rows, int32_t heads, int32_t head_dim,
                                      uint8_t* codes, float* scale, void* hip_stream) {
  clear_error();
  hsap_status st = check_quantize(x, groups, rows, heads, head_dim, codes, scale);
  if (st != HSAP_OK) return st;
  if ((int64_t)groups * heads > HSAP_QUANT_NOALLOC_MAX_SLICES)
    HSAP_FAIL(HSAP_ERR_UNSUPPORTED, "groups x heads = %lld above the scratch limit of %d slices",
              (long long)groups * heads, HSAP_QUANT_NOALLOC_MAX_SLICES);
  float* work = nullptr;
  st = scratch_for_current_device(&work);
  if (st != HSAP_OK) return st;
  return quantize(x, groups, rows, heads, head_dim, codes, scale, work, (hipStream_t)hip_stream);
}

hsap_status hsap_doc_start(const int32_t* cu_seqlens, int32_t num_docs, int64_t total_tokens, int32_t* doc_start,
                           void* hip_stream) {
  clear_error();
  if (!cu_seqlens || !doc_start) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (num_docs < 1) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "num_docs %d < 1", num_docs);
  if (total_tokens <= 0 || total_tokens > INT32_MAX) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "bad total_tokens");
  hipLaunchKernelGGL(doc_start_kernel, dim3(grid_for(total_tokens)), dim3(256), 0, (hipStream_t)hip_stream,
                     cu_seqlens, num_docs, total_tokens, doc_start);
  return check_launch("doc_start");
}

hsap_status hsap_shard_gather(const hsap_shard_desc* shard, const void* src, void* dst, int64_t row_bytes,
                              void* hip_stream) {
  clear_error();
  if (!shard) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "shard descriptor is NULL");
  hsap_shard_desc d = *shard;
  d.shard_id = 0;  // only N, P and the layout matter here
  d.block_m = d.block_n = 1;
  Geom g;
  hsap_status st = check_shard(&d, &g);
  if (st != HSAP_OK) return st;
  if (!src || !dst) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "NULL pointer argument");
  if (row_bytes <= 0 || row_bytes % 16) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "row_bytes must be a positive multiple of 16");
  if (((uintptr_t)src | (uintptr_t)dst) & 15) HSAP_FAIL(HSAP_ERR_INVALID_ARG, "src and dst must be 16-byte aligned");
  hipLaunchKernelGGL(gather_kernel, dim3(grid_for(g.N * (row_bytes / 16))), dim3(256), 0, (hipStream_t)hip_stream, g,
                     (const uint4*)src, (uint4*)dst, row_bytes / 16);
  return check_launch("shard_gather");
}

}  // extern "C"
