// Internal interface between the host runtime and the gfx950 kernels.
// Not part of the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vla {

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

// Most frames (robots' action phases) one skinny GEMM, norm or cache
// attention launch can carry as frame blocks.
constexpr int MAX_FRAMES = 8;

// GEMM epilogues. Physical output column n of a GEMM is row n of its weight
// matrix as stored on the device; paired kinds read columns n and n + 16 of
// every 32-column group together.
enum EpiKind {
  EPI_F32 = 0,   // out_f32[m, n] = v + bias[n] + rowadd[m % period, n]
  EPI_T,         // out_T[m, n] = T(v + bias[n])
  EPI_RESID,     // resid[m, n] += v + bias[n]                 (fp32 residual stream)
  EPI_GELU,      // out_T[m, n] = T(gelu_tanh(v + bias[n]))
  EPI_SWISH,     // out_T[m, n] = T(swish(v + bias[n]))
  EPI_GEGLU,     // gate/up interleaved in 16-row blocks: out_T[m, 16g+j] = T(gelu(gate) * up)
  EPI_QKV_ROPE,  // q/k rotated pairs (rotate-half, permuted rows), v plain; written to q / k / v
  EPI_QKV_PLAIN, // columns [q (nq*hd) | k (nkv*hd) | v (nkv*hd)] without rotation, any hd
  EPI_EULER,     // x[m, n] += dt * (v + bias[n]); xop[m, n] = T(x[m, n])
  EPI_PART,      // raw fp32 result into out = [splits][M][N] (ldo = its capacity in floats);
                 // the consumer sums the splits in order
};
// With Epi::afrag set, the operand-type outputs (out, xop) are written in
// the row-block operand layout (afrag_index) instead of row-major.

// KV-cache layout ("MFMA fragment order"). Keys go in blocks of 32; every
// 1 KB chunk holds exactly the 64 lanes x 16 bytes one MFMA operand load of
// the attention kernel reads, so those loads are contiguous. VEC is the
// elements per 16 bytes (8 bf16, 4 fp32), SW = 4 VEC the K-extent of one
// MFMA step. Per KV head j, nb blocks:
//  K (the A operand of S^T = K Q^T): chunk (block b, 16-key tile nt, d-slab
//    s of SW) = 64 lanes; lane (g, i) = 16 g + i holds d = s SW + g VEC ..
//    + VEC - 1 of the key in row i of tile nt, which is key
//    32 b + 8 (i / 4) + 4 nt + i % 4 (bf16) or 32 b + 16 nt + i (fp32), so
//    that a lane group's score rows are the keys of its P^T slice.
//  V (the A operand of O^T += V^T P^T): chunk (block b, 16-row d-tile dt,
//    key slab kk of SW) = 64 lanes; lane (g, i) holds keys
//    32 b + kk SW + g VEC .. + VEC - 1 of d = 16 dt + i.
// Elements outside [0, S) x [0, hd) are never written (buffers start zeroed;
// V there must stay zero, since a zero probability times a non-finite value
// would not vanish).
__host__ __device__ inline int kv_vec(int dtype) { return dtype == DT_BF16 ? 8 : 4; }
__host__ __device__ inline size_t kv_kidx(int dtype, int nb, int hd, int j, int key, int d) {
  const int vec = kv_vec(dtype), sw = 4 * vec, ns = (hd + sw - 1) / sw;
  const int b = key >> 5, kin = key & 31;
  const int nt = dtype == DT_BF16 ? (kin >> 2) & 1 : kin >> 4;
  const int i = dtype == DT_BF16 ? 4 * (kin >> 3) + (kin & 3) : kin & 15;
  const int s = d / sw, g = (d % sw) / vec, e = d % vec;
  return ((((size_t)j * nb + b) * 2 + nt) * ns + s) * 64 * vec + (size_t)(16 * g + i) * vec + e;
}
__host__ __device__ inline size_t kv_vidx(int dtype, int nb, int hd, int j, int key, int d) {
  const int vec = kv_vec(dtype), sw = 4 * vec, ndt = (hd + 15) / 16, pvs = 32 / sw;
  const int b = key >> 5, kin = key & 31;
  const int kk = kin / sw, g = (kin % sw) / vec, e = kin % vec;
  const int dt = d >> 4, i = d & 15;
  return ((((size_t)j * nb + b) * ndt + dt) * pvs + kk) * 64 * vec + (size_t)(16 * g + i) * vec + e;
}
// elements of one K or V buffer (all nkv heads)
inline size_t kv_kelems(int dtype, int nb, int hd, int nkv) {
  const int sw = 4 * kv_vec(dtype);
  return (size_t)nkv * nb * 32 * ((hd + sw - 1) / sw) * sw;
}
inline size_t kv_velems(int dtype, int nb, int hd, int nkv) {
  return (size_t)nkv * nb * 32 * ((hd + 15) / 16) * 16;
}

// Row-block operand layout of the skinny GEMM's A (at most 64 rows): chunk
// (K-slab ks of SW, 16-row tile mt) is 1 KB, lane (g, i) = 16 g + i holding
// row 16 mt + i, columns SW ks + g VEC .. + VEC - 1; chunks go K-slab-major,
// so the four row tiles of a slab are adjacent. Producers of such operands
// write it directly; every load of the skinny kernel is then contiguous.
__host__ __device__ inline size_t afrag_index(int dtype, int m, int k) {
  const int vec = kv_vec(dtype), sw = 4 * vec;
  const int lane = (m & 15) + 16 * ((k % sw) / vec);
  return (((size_t)(k / sw) * 4 + (m >> 4)) * 64 + lane) * vec + k % vec;
}
inline size_t afrag_elems(int dtype, int K) {
  const int sw = 4 * kv_vec(dtype);
  return (size_t)((K + sw - 1) / sw) * sw * 64;
}
// Frame blocks: an operand of several frames' rows (a batched action phase)
// holds each frame's blk_rows rows (<= 64) in its own row-block layout,
// blk_elems elements apart; blk_rows == 0 means one block (m < 64).
__host__ __device__ inline size_t afrag_index_blk(int dtype, int m, int k, int blk_rows, size_t blk_elems) {
  if (blk_rows <= 0) return afrag_index(dtype, m, k);
  return (size_t)(m / blk_rows) * blk_elems + afrag_index(dtype, m % blk_rows, k);
}

struct Epi {
  int kind = EPI_F32;
  int afrag = 0;
  void* out = nullptr;
  int ldo = 0;
  const float* bias = nullptr;
  const float* rowadd = nullptr;
  int rowadd_period = 1;
  int ldra = 0;
  float* resid = nullptr;
  int ldr = 0;
  // EPI_QKV_ROPE: q row-major [m][ldq]; k and v in the KV-cache layout
  // (kv_kidx / kv_vidx) with kv_nb 32-key blocks per KV head, row m = key m
  void* q = nullptr;
  int ldq = 0;
  void* k = nullptr;
  void* v = nullptr;
  int kv_nb = 0;
  int nq = 0, nkv = 0, hd = 0, pos0 = 0;
  const float* rope_cos = nullptr;  // [pos][hd/2]
  const float* rope_sin = nullptr;
  // EPI_EULER
  float* x = nullptr;
  int ldx = 0;
  void* xop = nullptr;
  int ldxop = 0;
  float dt = 0.f;
  float xs = 1.f;  // EPI_EULER: x <- xs x + dt v
  // Frame blocks (batched action phase): with blk_rows > 0, row m is row
  // m % blk_rows of frame m / blk_rows. Row-block-layout outputs (out, xop)
  // of frame b start b * blk_out elements in (see afrag_index_blk), its own
  // K / V b * blk_k / b * blk_v elements in, with that frame's rows as keys
  // and RoPE positions pos0 + m % blk_rows. Row-major outputs use row m.
  int blk_rows = 0;
  size_t blk_out = 0, blk_xop = 0, blk_k = 0, blk_v = 0;
  // RMSNorm folded across a split-K skinny GEMM and the next skinny GEMM
  // (one frame, M <= 64, N <= 64 x 32):
  // * producer (EPI_PART with norm_g set): the last split to arrive for a
  //   32-column pair sums the pair's partials in split order into the fp32
  //   residual x (ldx), writes norm_out = T(x * norm_g) (per column; in the
  //   row-block operand layout when afrag) and the pair's per-row sum of
  //   squares rowss[pair][m]. cnt: one counter per pair, zero before the
  //   first launch and left at zero;
  // * consumer (any other kind, rowss set): the product of each row m is
  //   scaled by 1 / sqrt(sum over the rowss_n pairs of rowss[pair][m] /
  //   rowss_d + 1e-6) before the epilogue; the pairs are summed in a fixed
  //   order. Since the scale is per row it commutes with the product, so
  //   the two launches compute the RMSNorm of x with gain norm_g followed
  //   by the GEMM, with T rounding before the scale instead of after.
  const float* norm_g = nullptr;
  void* norm_out = nullptr;
  float* rowss = nullptr;
  int rowss_n = 0, rowss_d = 0;
  unsigned* cnt = nullptr;
};

struct GemmDesc {
  int dtype;
  const void* A;
  int lda;
  const void* W;
  int ldw;
  int M, N, K;
  Epi epi;
  // Fragment-ordered weights (skinny kernel, M <= 64): K-slabs per n-block in
  // the stored tensor and the first slab used; frag_ks == 0 means row-major W.
  // With fragment-ordered weights A is in the row-block operand layout
  // (afrag_index) and lda is unused.
  int frag_ks = 0;
  int frag_ks0 = 0;
  // Skinny kernel only: `frames` row blocks of M rows each (a batched action
  // phase), block f of A at A + f * a_blk elements; the weights are loaded
  // once for all of them and every row is computed exactly as in a
  // one-frame call. The epilogue sees rows f * M + m (Epi::blk_rows = M).
  int frames = 1;
  size_t a_blk = 0;
  // Row count the split-K factor is planned for (0: M). A batched prefill
  // passes one frame's rows, so every row gets the same reduction as in a
  // one-frame call; batched action loops pass a fixed reference (the largest
  // group), so the reduction does not depend on the group size.
  int plan_m = 0;
  // The most plan_m-row blocks a launch of this plan stacks (a prefill
  // batch). The split count may then be planned for that launch as well
  // (fixed for every batch, so the reduction stays the same).
  int plan_batch = 1;
};

// Offset of element (n, k) of a weight stored in MFMA fragment order with KS
// K-slabs (of frag_slab(dtype) elements) per 16-row n-block.
size_t frag_index(int n, int k, int KS, int dtype);
int frag_slab(int dtype);

// Scratch the kernels may use (split-K and attention partials).
struct Scratch {
  float* ptr = nullptr;
  size_t floats = 0;
};

// Launch-size limits applied by the planner without changing any tile,
// split or reduction order (results are independent of them).
struct LaunchCaps {
  int max_wgs = 0;  // 0 = uncapped; otherwise grid-stride over tiles
  // when set, the main kernel of the launch records these at its own start
  // and end (measurement only)
  hipEvent_t ev_start = nullptr;
  hipEvent_t ev_stop = nullptr;
};

struct GemmPlan {
  int cfg;     // tile configuration index
  int splits;  // split-K factor
  int tiles;   // total tiles (incl. splits)
  size_t scratch_floats;
};

GemmPlan plan_gemm(const GemmDesc& g);
// Rows and columns of the tile of plan p (the skinny kernel: 0 rows, 32
// columns per workgroup).
void plan_tile(const GemmDesc& g, const GemmPlan& p, int* bm, int* bn);
hipError_t launch_gemm(const GemmDesc& g, const Scratch& s, const LaunchCaps& caps, hipStream_t st);

struct AttnDesc {
  int dtype;
  const void* q;  // [segs][Sq rows][ldq]
  int ldq;
  const void* k0;  // [segs][S0][ldkv]
  const void* v0;
  int S0;
  const void* k1;  // [segs][S1][ldkv] or null
  const void* v1;
  int S1;
  int ldkv;
  void* out;  // [segs][Sq][ldo]
  int ldo;
  int Sq, nq, nkv, hd;
  int segs;  // independent segments (camera views) with their own Q/K/V rows
  long long seg_q, seg_kv, seg_o;  // element strides between segments
  // segments of one frame when several frames' views are stacked: the KV
  // split is planned for plan_segs segments, so every segment is reduced
  // as in a one-frame call (0: plan for segs)
  int plan_segs = 0;
};

size_t attn_scratch_floats(const AttnDesc& a);

// Attention over keys [k0 (S0 keys); k1 (S1 keys)], both in the KV-cache
// layout with ceil(S / 32) blocks per KV head (see kv_kidx / kv_vidx). q and
// out row-major as in AttnDesc (one segment). No scratch.
struct AttnKvDesc {
  int dtype;
  const void* q;
  int ldq;
  const void* k0;
  const void* v0;
  int S0;
  const void* k1;
  const void* v1;
  int S1;
  void* out;
  int ldo;
  int out_afrag;  // out in the row-block operand layout (Sq <= 64), ldo unused
  int Sq, nq, nkv, hd;
  // Several frames in one launch (batched action phase): frame f has queries
  // q + f Sq ldq, keys [k0f[f] (S0); k1 + f k1_blk (S1)] (values alike) and
  // output out + f out_blk; frame 0 uses k0 / v0.
  int frames = 1;
  const void* k0f[MAX_FRAMES] = {};
  const void* v0f[MAX_FRAMES] = {};
  size_t k1_blk = 0, v1_blk = 0, out_blk = 0;
  // Room for key splits (optional): with part (part_floats floats) and cnt
  // (cnt_n counters, zero before the first launch; every launch leaves them
  // zero) a query tile's key blocks are split over several workgroups (at
  // most one block per wave each) whose partials the last one to finish
  // merges in split order. Without it each tile is one workgroup. The
  // result does not depend on the arrival order, only on the split count,
  // which depends on the shapes alone. Launches sharing part / cnt must not
  // overlap.
  float* part = nullptr;
  size_t part_floats = 0;
  unsigned* cnt = nullptr;
  int cnt_n = 0;
};
hipError_t launch_attention_kv(const AttnKvDesc& d, const LaunchCaps& caps, hipStream_t st);
// Floats of partials (and, in *counters, the counters) a launch of these
// shapes needs for its key splits; 0 when it runs unsplit.
size_t attn_kv_split_floats(int dtype, int frames, int Sq, int nq, int nkv, int hd, int S0, int S1, int* counters);
hipError_t launch_attention(const AttnDesc& a, const Scratch& s, const LaunchCaps& caps, hipStream_t st);

// Residual add + row norm: x[m] += bias + colscale * sum_s part[s][m] (split
// order; nothing is added when splits is 0, colscale NULL means 1), stored
// back, then out[m] = LayerNorm (biased variance) or RMSNorm of x[m], times
// gain (g, or 1 + g when g_plus_one) plus b, in the operand type: row-major
// with ldo, the row-block operand layout (afrag, rows <= 64 per frame block), or pixel
// shuffled (shuffle > 1: row = view * tview + y * grid_w + x of a raster
// patch grid goes to coarse row view * tview / s^2 + (y / s) * (grid_w / s)
// + x / s, columns offset by ((y % s) * s + x % s) * d; ldo = s^2 d).
// d <= 2048.
struct NormDesc {
  int dtype = DT_F32;
  float* x = nullptr;
  int ldx = 0, rows = 0, d = 0;
  const float* part = nullptr;
  int splits = 0;
  const float* bias = nullptr;
  const float* colscale = nullptr;
  const float* g = nullptr;
  int g_plus_one = 0;
  const float* b = nullptr;
  int rms = 0;
  void* out = nullptr;
  int ldo = 0;
  int afrag = 0;
  int shuffle = 1, grid_w = 0, tview = 0;
  int blk_rows = 0;     // afrag output in frame blocks (afrag_index_blk)
  size_t blk_out = 0;
};
hipError_t launch_norm(const NormDesc& n, hipStream_t st);

// Image [views][H][W][3] fp32 -> patches [views * T][ldo] of the operand type,
// columns beyond 3 p^2 zero.
hipError_t launch_patchify(int dtype, const float* pix, int views, int H, int W, int p, void* out,
                           int ldo, hipStream_t st);

// x[i, :] = E[ids[i], :] * scale (E [vocab, d] in the operand type; ids
// outside [0, vocab) are clamped).
hipError_t launch_embed(int dtype, const void* E, int d, int vocab, const int32_t* ids, int n,
                        float scale, float* x, int ldx, hipStream_t st);

// dst_T[r, c] = T(src[r, c]) for c < cols, 0 for cols <= c < ld_dst (row-major
// with ld_dst, or the row-block operand layout with K = ld_dst when afrag,
// in frame blocks of blk_rows rows blk_elems apart when blk_rows > 0);
// optionally also copies src into dst_f32 (fp32, ld = cols).
hipError_t launch_cvt_pad(int dtype, const float* src, int rows, int cols, void* dst, int ld_dst,
                          bool afrag, float* dst_f32, hipStream_t st, int blk_rows = 0,
                          size_t blk_elems = 0);

// Row-major copy of a weight stored in MFMA fragment order: out[n * K + k] =
// W[frag_index(n, k, KS)] for n < N, k < K (operand type; K a multiple of 8).
hipError_t launch_unfrag(int dtype, const void* frag, int N, int K, int KS, void* out, hipStream_t st);
// Device-to-device copy of `bytes` bytes as a kernel on stream st. (The
// runtime's device-to-device copies run as its own copy kernels, which a
// kernel trace shows on the default stream's hardware queue; this keeps the
// pipeline's staging copies on the queue of the stream that orders them.)
hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t st);

// dst[r, :] = row (operand type) for every r < rows.
hipError_t launch_bcast_row(int dtype, const void* row, int cols, void* dst, int ld_dst, int rows,
                            hipStream_t st);

// Per-workgroup residency log (measurement only). While a log is set, the
// first lane of every workgroup of the instrumented kernels appends one
// record when the workgroup starts and one when it ends: the time on the
// 100 MHz constant clock, the hardware-id register (CU, shader array and
// engine, and the queue the work came from), the XCC id, the kernel kind
// and whether it is the end.
struct WaveRec {
  uint64_t t;
  uint32_t hwid, xcc, kind, end;
};
// Eight slices (one per XCC, counters 256 bytes apart to keep the atomics
// of different XCCs off one cache line), cap records each.
constexpr int WAVELOG_SLICES = 8;
struct WaveLog {
  uint32_t cap, pad[63];
  uint32_t count[WAVELOG_SLICES * 64];  // slice x counts at count[64 x]
  WaveRec rec[1];                        // WAVELOG_SLICES * cap records follow
};
enum KernelKind {
  KK_GEMM = 1, KK_SPLITK, KK_SKINNY, KK_ATTN, KK_ATTN_COMBINE, KK_ATTN2, KK_NORM,
  KK_PATCHIFY, KK_EMBED, KK_CVT
};
// Point the kernels at a log (nullptr: off). Not while kernels run.
hipError_t wavelog_set(WaveLog* dev);

}  // namespace vla
