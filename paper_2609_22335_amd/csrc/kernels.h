// Internal interface between the host runtime and the gfx950 kernels.
// Not part of the C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vla {

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

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
  EPI_EULER,     // x[m, n] += dt * (v + bias[n]); xop[m, n] = T(x[m, n])
  EPI_PART,      // raw fp32 result into out = [splits][M][N] (ldo = its capacity in floats);
                 // the consumer sums the splits in order
};

struct Epi {
  int kind = EPI_F32;
  void* out = nullptr;
  int ldo = 0;
  const float* bias = nullptr;
  const float* rowadd = nullptr;
  int rowadd_period = 1;
  int ldra = 0;
  float* resid = nullptr;
  int ldr = 0;
  // EPI_QKV_ROPE
  void* q = nullptr;
  int ldq = 0;
  void* k = nullptr;
  void* v = nullptr;
  int ldkv = 0;
  int ldvt = 0;  // > 0: V is stored transposed, element (m, c) at v[c * ldvt + m]
  int nq = 0, nkv = 0, hd = 0, pos0 = 0;
  const float* rope_cos = nullptr;  // [pos][hd/2]
  const float* rope_sin = nullptr;
  // EPI_EULER
  float* x = nullptr;
  int ldx = 0;
  void* xop = nullptr;
  int ldxop = 0;
  float dt = 0.f;
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
  int frag_ks = 0;
  int frag_ks0 = 0;
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
};

size_t attn_scratch_floats(const AttnDesc& a);

// Attention over keys [k0 (S0 rows); k1 (S1 rows)] with V stored transposed:
// vt0 [n_kv * hd][ldvt0 >= round32(S0)], vt1 [n_kv * hd][ldvt1 >= round32(S1)],
// padding columns zero. K rows have ldk elements (head j at column j * hd).
// q and out as in AttnDesc (one segment). No scratch.
struct AttnVtDesc {
  int dtype;
  const void* q;
  int ldq;
  const void* k0;
  const void* vt0;
  int S0, ldvt0;
  const void* k1;
  const void* vt1;
  int S1, ldvt1;
  int ldk;
  void* out;
  int ldo;
  int Sq, nq, nkv, hd;
};
hipError_t launch_attention_vt(const AttnVtDesc& d, const LaunchCaps& caps, hipStream_t st);
hipError_t launch_attention(const AttnDesc& a, const Scratch& s, const LaunchCaps& caps, hipStream_t st);

// Residual add + row norm: x[m] += bias + sum_s part[s][m] in split order
// (part [splits][rows][d]; nothing is added when splits is 0), then
// out[m] = LayerNorm (biased variance) or RMSNorm of x[m], times g (+ b),
// in the operand type. d <= 2048.
hipError_t launch_norm(int dtype, float* x, int ldx, int rows, int d, const float* part,
                       int splits, const float* bias, const float* g, const float* b, bool rms,
                       void* out, int ldo, hipStream_t st);

// Image [views][H][W][3] fp32 -> patches [views * T][ldo] of the operand type,
// columns beyond 3 p^2 zero.
hipError_t launch_patchify(int dtype, const float* pix, int views, int H, int W, int p, void* out,
                           int ldo, hipStream_t st);

// x[i, :] = E[ids[i], :] * scale (E [vocab, d] in the operand type; ids
// outside [0, vocab) are clamped).
hipError_t launch_embed(int dtype, const void* E, int d, int vocab, const int32_t* ids, int n,
                        float scale, float* x, int ldx, hipStream_t st);

// dst_T[r, c] = T(src[r, c]) for c < cols, 0 for cols <= c < ld_dst;
// optionally also copies src into dst_f32 (fp32, ld = cols).
hipError_t launch_cvt_pad(int dtype, const float* src, int rows, int cols, void* dst, int ld_dst,
                          float* dst_f32, hipStream_t st);

// dst[r, :] = row (operand type) for every r < rows.
hipError_t launch_bcast_row(int dtype, const void* row, int cols, void* dst, int ld_dst, int rows,
                            hipStream_t st);

}  // namespace vla
