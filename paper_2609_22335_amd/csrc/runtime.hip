// Host runtime and C ABI of the two-phase VLA library (see include/vla.h).
//
// Phase 1 (VLM prefill) and phase 2 (flow-matching action denoising) are
// sequences of kernel launches on a caller-given stream. The pipeline runs
// frame r's action phase on one stream while frame r+1's prefill runs on a
// second one (the cross-frame pipelining of Section 2.1), with two model-owned
// contexts so the prefill of frame r+1 never overwrites the cache frame r is
// still reading.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/vla.h"
#include "gen.h"
#include "kernels.h"

using namespace vla;

// ---------------------------------------------------------------------------
// Errors
// ---------------------------------------------------------------------------

static thread_local std::string g_err;

static int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess)                                                               \
      return fail(VLA_EHIP, std::string(#expr) + ": " + hipGetErrorString(e_));         \
  } while (0)

#define VLA_TRY(expr)            \
  do {                           \
    int r_ = (expr);             \
    if (r_ != VLA_OK) return r_; \
  } while (0)

static inline int rnd_up(int x, int m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------------------
// Configuration
// ---------------------------------------------------------------------------

struct Dims {
  int gh, gw, tview, nimg, prefix, kp, kp_pad, a_pad, s_pad, rows_v, kvd, qd, qkv_n, vhd;
  int kproj;  // projector input width (ViT width times the pixel-shuffle factor squared)
  int ehd;    // DiT head dim
  int prefix_pad, chunk_pad;  // key lengths rounded up to 32 (KV-cache blocks)
  int arows;  // rows of the action head's token sequence (chunk, plus the cognition and time tokens)
};

static Dims derive(const vla_config& c) {
  Dims d{};
  d.gh = c.img_h / c.patch;
  d.gw = c.img_w / c.patch;
  d.tview = d.gh * d.gw;
  d.nimg = c.n_views * d.tview / (c.shuffle * c.shuffle);
  d.prefix = d.nimg + c.n_text + (c.state_dim > 0 ? 1 : 0) + (c.head == VLA_HEAD_COG ? 1 : 0);
  d.kp = 3 * c.patch * c.patch;
  d.kp_pad = rnd_up(d.kp, 8);
  d.a_pad = rnd_up(c.action_dim, 8);
  d.s_pad = rnd_up(std::max(c.state_dim, 1), 8);
  d.rows_v = c.n_views * d.tview;
  d.kproj = c.vit_dim * c.shuffle * c.shuffle;
  d.ehd = c.head != VLA_HEAD_PI0 ? c.ex_dim / c.ex_heads : c.head_dim;
  d.kvd = c.lm_kv_heads * c.head_dim;
  d.qd = c.lm_heads * c.head_dim;
  d.qkv_n = d.qd + 2 * d.kvd;
  d.vhd = c.vit_dim / c.vit_heads;
  d.prefix_pad = rnd_up(d.prefix, 32);
  d.arows = c.chunk_len + (c.head == VLA_HEAD_COG ? 2 : 0);
  d.chunk_pad = rnd_up(d.arows, 32);
  return d;
}

static int validate(const vla_config* c) {
  if (!c) return fail(VLA_EINVAL, "config is NULL");
  auto bad = [](const char* what) { return fail(VLA_EINVAL, std::string("invalid config: ") + what); };
  if (c->dtype != VLA_F32 && c->dtype != VLA_BF16) return bad("dtype");
  const int pos[] = {c->n_views, c->img_h, c->img_w, c->patch, c->vit_dim, c->vit_heads, c->vit_mlp,
                     c->vit_layers, c->lm_dim, c->lm_heads, c->lm_kv_heads, c->head_dim, c->lm_mlp,
                     c->lm_layers, c->vocab, c->ex_dim, c->ex_mlp, c->ex_layers, c->chunk_len,
                     c->action_dim, c->n_steps};
  for (int v : pos)
    if (v <= 0) return bad("every size except n_text and state_dim must be positive");
  if (c->n_text < 0 || c->state_dim < 0) return bad("n_text / state_dim negative");
  if (c->img_h % c->patch || c->img_w % c->patch) return bad("patch must divide the image");
  if (c->vit_dim % c->vit_heads) return bad("vit_heads must divide vit_dim");
  const int vhd = c->vit_dim / c->vit_heads;
  if (vhd % 8 || vhd > 256) return bad("ViT head dim must be a multiple of 8 and <= 256");
  if (c->lm_heads % c->lm_kv_heads) return bad("lm_heads % lm_kv_heads != 0");
  if (c->head_dim % 32 || c->head_dim > 256) return bad("head_dim must be a multiple of 32, <= 256");
  if (c->dtype == VLA_F32 && (c->head_dim > 128 || vhd > 128))
    return bad("fp32 configurations need head dims <= 128");
  if (c->head != VLA_HEAD_PI0 && c->head != VLA_HEAD_DIT && c->head != VLA_HEAD_COG) return bad("head");
  if (c->shuffle < 1 || (c->img_h / c->patch) % c->shuffle || (c->img_w / c->patch) % c->shuffle)
    return bad("shuffle must be >= 1 and divide the patch grid");
  if (c->head == VLA_HEAD_PI0) {
    if (c->ex_layers != c->lm_layers) return bad("ex_layers must equal lm_layers (layer-wise KV sharing)");
  } else {
    if (c->head == VLA_HEAD_COG && c->chunk_len > 62)
      return bad("cognition-token head: chunk_len + 2 tokens must be <= 64");
    if (c->ex_heads <= 0 || c->ex_dim % c->ex_heads) return bad("ex_heads must divide ex_dim");
    const int ehd = c->ex_dim / c->ex_heads;
    if (ehd % 8 || ehd > 256 || (c->dtype == VLA_F32 && ehd > 128))
      return bad("DiT head dim must be a multiple of 8, <= 256 (<= 128 in fp32)");
    if (c->ex_dim % 2) return bad("ex_dim must be even");
  }
  if (c->lm_mlp % 16 || c->ex_mlp % 16) return bad("lm_mlp / ex_mlp must be multiples of 16");
  if (c->vit_dim % 8 || c->lm_dim % 8 || c->ex_dim % 8 || c->vit_mlp % 8)
    return bad("model widths must be multiples of 8");
  if (c->ex_dim % 32) return bad("ex_dim must be a multiple of 32");
  if (c->chunk_len > 64 || c->n_steps > 64) return bad("chunk_len and n_steps must be <= 64");
  if (c->sampler != VLA_SAMPLER_EULER && c->sampler != VLA_SAMPLER_DDIM) return bad("unknown sampler");
  if (c->sampler == VLA_SAMPLER_DDIM && c->n_steps > 1000) return bad("DDIM: n_steps must be <= 1000");
  return VLA_OK;
}

static bool preset(const char* name, vla_config* o) {
  if (!name || !o) return false;
  const std::string n(name);
  if (n == "tiny" || n == "tiny_ddim") {
    *o = vla_config{VLA_F32, 1, 128, 128, 16, 256, 4, 1024, 2, 256, 4, 1, 64, 1024, 2,
                    1024, 16, 0, 128, 512, 2, 8, 7, 4, VLA_HEAD_PI0, 1, 0, VLA_SAMPLER_EULER};
    if (n == "tiny_ddim") o->sampler = VLA_SAMPLER_DDIM;
    return true;
  }
  if (n == "tiny_dit") {
    *o = vla_config{VLA_F32, 1, 128, 128, 16, 256, 4, 1024, 2, 256, 4, 4, 64, 1024, 2,
                    1024, 16, 0, 192, 768, 4, 8, 7, 4, VLA_HEAD_DIT, 2, 4};
    return true;
  }
  if (n == "gr00t") {
    *o = vla_config{VLA_BF16, 1, 448, 448, 28, 1152, 16, 4304, 27, 2048, 16, 16, 128, 8192, 12,
                    1024, 32, 0, 1536, 6144, 16, 16, 32, 4, VLA_HEAD_DIT, 2, 32};
    return true;
  }
  if (n == "cogact" || n == "tiny_cog") {
    if (n == "cogact")
      *o = vla_config{VLA_BF16, 1, 224, 224, 14, 1152, 16, 4304, 27, 2048, 8, 1, 256, 16384, 18,
                      1024, 48, 0, 1024, 4096, 24, 16, 7, 10, VLA_HEAD_COG, 1, 16, VLA_SAMPLER_DDIM};
    else
      *o = vla_config{VLA_F32, 1, 128, 128, 16, 256, 4, 1024, 2, 256, 4, 1, 64, 1024, 2,
                      1024, 16, 0, 128, 512, 2, 8, 7, 4, VLA_HEAD_COG, 1, 2, VLA_SAMPLER_DDIM};
    return true;
  }
  if (n == "pi0" || n == "pi0_3view" || n == "pi0_ddim") {
    *o = vla_config{VLA_BF16, 1, 224, 224, 14, 1152, 16, 4304, 27, 2048, 8, 1, 256, 16384, 18,
                    1024, 48, 32, 1024, 4096, 18, 50, 32, 10, VLA_HEAD_PI0, 1, 0, VLA_SAMPLER_EULER};
    if (n == "pi0_3view") {
      o->n_views = 3;
      o->n_text = 64;
    }
    if (n == "pi0_ddim") o->sampler = VLA_SAMPLER_DDIM;
    return true;
  }
  return false;
}

// ---------------------------------------------------------------------------
// Parameters: logical tensors (names and [out, in] shapes of the inventory)
// placed into device tensors with a row map.
// ---------------------------------------------------------------------------

enum RowMap { MAP_IDENT = 0, MAP_ROPE, MAP_GATE, MAP_UP };
constexpr int DIT_TIME_DIM = 256;  // width of the DiT's sinusoidal timestep embedding

struct DevTensor {
  size_t offset = 0;  // into the weight arena
  int rows = 0, ld = 0, dt = DT_F32;
  bool vec = false;  // fp32 vector: params sit at column offsets (row_off) of one row
  int fks = 0;       // > 0: MFMA fragment order with fks K-slabs per 16-row block
  size_t bytes() const {
    const size_t e = dt == DT_BF16 ? 2 : 4;
    if (fks > 0) return (size_t)((rows + 31) / 32 * 32) * fks * frag_slab(dt) * e;
    return (size_t)rows * ld * e;
  }
  size_t index(int r, int c) const {
    return fks > 0 ? frag_index(r, c, fks, dt) : (size_t)r * ld + c;
  }
};

struct ParamRec {
  std::string name;
  int rows, cols;
  double mean, stdv;
  int tensor;  // index into model tensors
  int map, row_off, hd;
};

static int dev_row(const ParamRec& p, int r) {
  switch (p.map) {
    case MAP_ROPE: {
      const int head = r / p.hd, i = r % p.hd, half = p.hd / 2;
      const int ph = i < half ? 32 * (i / 16) + i % 16 : 32 * ((i - half) / 16) + 16 + (i - half) % 16;
      return p.row_off + head * p.hd + ph;
    }
    case MAP_GATE: return p.row_off + 32 * (r / 16) + r % 16;
    case MAP_UP: return p.row_off + 32 * (r / 16) + 16 + r % 16;
    default: return p.row_off + r;
  }
}

struct VitLayer {
  int ln1_g, ln1_b, qkv_w, qkv_b, o_w, o_b, ln2_g, ln2_b, fc1_w, fc1_b, fc2_w, fc2_b;
};
struct DecLayer {
  int rms1, qkv, o, rms2, gu, down;  // tensor ids (-1 when absent)
};
// DiT layer: cross layers (even) have q and kv (row-major, features -> K|V),
// self layers (odd) a fused q|k|v.
struct DitLayer {
  int ada_w = -1, ada_b = -1, q = -1, kv = -1, qkv = -1, o = -1, fc1 = -1, fc2 = -1;
};

// Cognition-token head layer: pre-LN self-attention (fused q|k|v, no
// biases) and GELU MLP.
struct CogLayer {
  int ln1_g = -1, ln1_b = -1, qkv = -1, o = -1, ln2_g = -1, ln2_b = -1, fc1 = -1, fc2 = -1;
};

constexpr int MAX_ACT_STREAMS = 4;

constexpr int MAX_VLM_STREAMS = 2;
constexpr int MAX_ACT_BATCH = MAX_FRAMES;  // frames one action phase can run together

struct Streams {
  hipStream_t v[MAX_VLM_STREAMS] = {};
  hipStream_t a[MAX_ACT_STREAMS] = {};
};

constexpr int MAX_VLM_BATCH = 8;  // frames one prefill can run together
constexpr int CTX_BLOCK = 8;      // pipeline contexts are allocated in blocks of this many

// Scratch of one VLM lane (one prefill at a time per lane), with staging for
// graph replays, sized for `cap` frames prefilled together (each buffer holds
// the frames' rows one after another).
struct VlmWs {
  int cap = 1;
  float *xv = nullptr, *xl = nullptr;
  void *h = nullptr, *qkv = nullptr, *att = nullptr, *mlp = nullptr, *sbuf = nullptr;
  Scratch scr;
  float* pstage = nullptr;
  int32_t* istage = nullptr;
  float* sstage = nullptr;
  std::vector<void*> mem;  // this lane's allocations
  ~VlmWs() {
    for (void* p : mem) hipFree(p);
  }
};

// Scratch of one action lane (one denoise at a time per lane).
// Action-phase workspace, sized for MAX_ACT_BATCH frames: row-major buffers
// hold the frames' rows one after another; row-block-layout operands hold
// one block per frame, the blk_* elements apart.
struct ActWs {
  float* u = nullptr;
  void *xop = nullptr, *a = nullptr, *hid = nullptr, *h = nullptr, *q = nullptr;
  void *kown = nullptr, *vown = nullptr, *att = nullptr, *mlp = nullptr;
  float* xg = nullptr;      // chunks written by graph replays, copied out afterwards
  float* nstage = nullptr;  // noise staged for graph replays
  // key-split partials and counters of the cache attention (counters zero
  // between launches)
  float* apart = nullptr;
  size_t apart_floats = 0;
  unsigned* acnt = nullptr;
  int acnt_n = 0;
  // one-frame expert layers fold each RMSNorm into the GEMMs around it
  // (Epi::rowss): the per-pair row sums of squares [pair][row] and the pair
  // counters of the split-K producers (zero between launches)
  float* rowss = nullptr;
  unsigned* pcnt = nullptr;
  size_t blk_xop = 0, blk_de = 0, blk_att = 0, blk_mlp = 0, blk_k = 0, blk_v = 0;
  Scratch scr;
};
constexpr int FOLD_MAX_PAIRS = 64;  // expert width <= 64 x 32

struct vla_ctx {
  vla_model* m = nullptr;
  // contexts made together share one allocation per buffer (context i of a
  // block at i times the context size); the block's first context owns it
  bool own = true;
  // per layer, the KV-cache layout (kv_kidx / kv_vidx) with prefix_pad / 32
  // blocks per KV head; zeroed at creation, so unwritten padding stays zero
  void* K = nullptr;
  void* V = nullptr;
  // DiT head: cross K/V of every even DiT layer (same layout, ex_heads heads)
  void* XK = nullptr;
  void* XV = nullptr;
  // cognition-token head: the conditioning vector c = W_c f + b_c, fp32 [ex_dim]
  float* cog = nullptr;
};

struct vla_model {
  vla_config c{};
  Dims d{};
  int dt = DT_F32;
  size_t esz = 4;
  int device = 0, num_cus = 0;
  uint64_t seed = 0;

  void* arena = nullptr;
  size_t arena_bytes = 0;
  std::vector<DevTensor> T;
  std::vector<ParamRec> P;
  std::map<std::string, int> pidx;

  // tensor ids
  int patch_w, patch_b, pos, post_g, post_b, proj_w, proj_b, embed, state_w = -1, state_b = -1;
  std::vector<VitLayer> vit;
  std::vector<DecLayer> lm, ex;
  int in_w, in_b, t1_w, t1_b, t2_w, t2_b, fin_g = -1, out_w, out_b;
  // DiT head
  int lm_fin_g = -1, fada_w = -1, fada_b = -1;
  std::vector<DitLayer> dit;
  // cognition-token head: the token row, its projection, the head's layers,
  // the final LayerNorm bias and the time token of every step [n_steps][ex_dim]
  int cog_tok = -1, cog_w = -1, cog_b = -1, fin_b = -1;
  std::vector<CogLayer> cogl;
  float* ttok = nullptr;

  // constant tables
  float* rope_cos = nullptr;
  float* rope_sin = nullptr;
  void* phi = nullptr;  // [n_steps][ex_dim] operand type, row-block operand layout
  float* ck = nullptr;  // [n_steps][ex_dim]: W_2 phi(t_k) + b_2
  // per step k: x <- step_a[k] x + step_b[k] v (Euler: 1 and -1/N; DDIM:
  // a_k and b_k of the header), and the head's time input t_k
  std::vector<float> step_a, step_b, step_t;
  // DiT head: adaLN vectors per step, [n_steps][ex_layers][6][ex_dim]
  // (shift1, scale1, gate1, shift2, scale2, gate2), final [n_steps][2][ex_dim]
  // (shift, scale), token positions [chunk_len][ex_dim]
  float* ada = nullptr;
  float* fada = nullptr;
  float* dpos = nullptr;

  // Row-major copies of the expert layers' matrices (qkv, o, gate/up, down)
  // for batched action loops, made on first use from the fragment-ordered
  // weights; one allocation.
  struct WideLayer {
    const void *qkv = nullptr, *o = nullptr, *gu = nullptr, *down = nullptr;
  };
  std::vector<WideLayer> exw;
  void* exw_mem = nullptr;

  // phase scratch
  std::vector<std::unique_ptr<VlmWs>> vws;  // VLM lanes; lane 0 serves standalone calls
  WaveLog* wlog = nullptr;                  // residency log (measurement), device memory
  size_t wlog_cap = 0;
  std::vector<std::unique_ptr<ActWs>> aws;  // action lanes; lane 0 serves standalone calls
  // Standalone calls share lane 0 of their phase (0: prefill, 1: denoise):
  // the stream and completion event of the last one, so that a call on
  // another stream first waits for it.
  struct Solo {
    hipEvent_t done = nullptr;
    hipStream_t stream = nullptr;
    bool pending = false;
  } solo[2];
  std::vector<void*> allocs;

  // pipeline
  std::vector<vla_ctx*> pctx;  // ring of act_streams + 1 contexts
  std::map<std::pair<int, int>, Streams> mask_streams;
  Streams plain{};
  std::vector<hipEvent_t> ev;   // per frame: VLM start, end
  std::vector<hipEvent_t> eva;  // per action item: start, end
  // graph replay: frame inputs staged into fixed buffers, graphs cached per
  // (context, VLM grid cap) and (action lane, context)
  std::map<std::tuple<int, int, int, int>, hipGraphExec_t> pre_graphs;  // (VLM lane, first context, WG cap, frames)
  std::map<std::pair<int, std::vector<int>>, hipGraphExec_t> den_graphs;  // (lane, contexts of the items)
  std::mutex mu;

  // per-tag kernel timer: every launch whose tag matches is bracketed by
  // events on its own stream
  std::string timer_tag;
  std::vector<hipEvent_t> timer_ev;  // pairs (begin, end)
  size_t timer_used = 0;

  char* tptr(int t) const { return (char*)arena + T[t].offset; }
  float* f32(int t) const { return (float*)tptr(t); }
};

// elements per layer of a context's K and V, and of an action lane's own K, V
static size_t ctx_layer_k(const vla_model* m) {
  return kv_kelems(m->dt, m->d.prefix_pad / 32, m->c.head_dim, m->c.lm_kv_heads);
}
static size_t ctx_layer_v(const vla_model* m) {
  return kv_velems(m->dt, m->d.prefix_pad / 32, m->c.head_dim, m->c.lm_kv_heads);
}
static int own_heads(const vla_model* m) {
  return m->c.head != VLA_HEAD_PI0 ? m->c.ex_heads : m->c.lm_kv_heads;
}
static size_t own_k(const vla_model* m) {
  return kv_kelems(m->dt, m->d.chunk_pad / 32, m->d.ehd, own_heads(m));
}
static size_t own_v(const vla_model* m) {
  return kv_velems(m->dt, m->d.chunk_pad / 32, m->d.ehd, own_heads(m));
}
// one even DiT layer's cross K or V (prefix keys, ex_heads heads)
static size_t cross_elems(const vla_model* m) {
  return std::max(kv_kelems(m->dt, m->d.prefix_pad / 32, m->d.ehd, m->c.ex_heads),
                  kv_velems(m->dt, m->d.prefix_pad / 32, m->d.ehd, m->c.ex_heads));
}

// bytes of one context's K, V and DiT cross K / V buffers
static size_t ctx_kbytes(const vla_model* m) { return (size_t)m->c.lm_layers * ctx_layer_k(m) * m->esz; }
static size_t ctx_vbytes(const vla_model* m) { return (size_t)m->c.lm_layers * ctx_layer_v(m) * m->esz; }
static size_t ctx_xbytes(const vla_model* m) {
  return m->c.head == VLA_HEAD_DIT ? (size_t)((m->c.ex_layers + 1) / 2) * cross_elems(m) * m->esz : 0;
}

// True when c[0 .. n-1] are consecutive contexts of one block.
static bool ctx_consecutive(const vla_model* m, vla_ctx* const* c, int n) {
  for (int i = 1; i < n; ++i)
    if (c[i]->K != (char*)c[0]->K + i * ctx_kbytes(m) || c[i]->V != (char*)c[0]->V + i * ctx_vbytes(m) ||
        c[i]->XK != (ctx_xbytes(m) ? (char*)c[0]->XK + i * ctx_xbytes(m) : nullptr))
      return false;
  return true;
}

static size_t dsz(int dt) { return dt == DT_BF16 ? 2 : 4; }

static int add_tensor(vla_model* m, int rows, int ld, int dt, bool vec = false, bool frag = false) {
  DevTensor t;
  t.rows = rows;
  t.ld = ld;
  t.dt = dt;
  t.vec = vec;
  if (frag) t.fks = (ld + frag_slab(dt) - 1) / frag_slab(dt);
  m->T.push_back(t);
  return (int)m->T.size() - 1;
}

static void add_param(vla_model* m, const std::string& name, int rows, int cols, double mean,
                      int tensor, int map = MAP_IDENT, int row_off = 0, int hd = 0) {
  ParamRec p{name, rows, cols, mean, 0.02, tensor, map, row_off, hd};
  m->pidx[name] = (int)m->P.size();
  m->P.push_back(p);
}

// Weight matrix [rows, cols] of the operand type, K padded to 8; `frag`
// stores it in MFMA fragment order for the skinny (M <= 64) GEMM.
static int add_mat(vla_model* m, const std::string& name, int rows, int cols, bool frag = false) {
  const int t = add_tensor(m, rows, rnd_up(cols, 8), m->dt, false, frag);
  add_param(m, name, rows, cols, 0.0, t);
  return t;
}
// fp32 vector (biases, norm gains: mean 1).
static int add_vec(vla_model* m, const std::string& name, int n, double mean = 0.0) {
  const int t = add_tensor(m, 1, n, DT_F32, true);
  add_param(m, name, 1, n, mean, t);
  return t;
}

static void build_inventory(vla_model* m) {
  const vla_config& c = m->c;
  const Dims& d = m->d;
  m->patch_w = add_mat(m, "vit.patch.w", c.vit_dim, d.kp);
  m->patch_b = add_vec(m, "vit.patch.b", c.vit_dim);
  m->pos = add_tensor(m, d.tview, c.vit_dim, DT_F32);
  add_param(m, "vit.pos", d.tview, c.vit_dim, 0.0, m->pos);
  for (int l = 0; l < c.vit_layers; ++l) {
    const std::string p = "vit." + std::to_string(l) + ".";
    VitLayer L{};
    L.ln1_g = add_vec(m, p + "ln1.g", c.vit_dim, 1.0);
    L.ln1_b = add_vec(m, p + "ln1.b", c.vit_dim);
    L.qkv_w = add_tensor(m, 3 * c.vit_dim, c.vit_dim, m->dt);
    L.qkv_b = add_tensor(m, 1, 3 * c.vit_dim, DT_F32, true);
    const char* qkv[3] = {"q", "k", "v"};
    for (int i = 0; i < 3; ++i) {
      add_param(m, p + qkv[i] + ".w", c.vit_dim, c.vit_dim, 0.0, L.qkv_w, MAP_IDENT, i * c.vit_dim);
      // biases live in one fp32 row; row_off counts columns for vectors
      add_param(m, p + qkv[i] + ".b", 1, c.vit_dim, 0.0, L.qkv_b, MAP_IDENT, i * c.vit_dim);
    }
    L.o_w = add_mat(m, p + "o.w", c.vit_dim, c.vit_dim);
    L.o_b = add_vec(m, p + "o.b", c.vit_dim);
    L.ln2_g = add_vec(m, p + "ln2.g", c.vit_dim, 1.0);
    L.ln2_b = add_vec(m, p + "ln2.b", c.vit_dim);
    L.fc1_w = add_mat(m, p + "fc1.w", c.vit_mlp, c.vit_dim);
    L.fc1_b = add_vec(m, p + "fc1.b", c.vit_mlp);
    L.fc2_w = add_mat(m, p + "fc2.w", c.vit_dim, c.vit_mlp);
    L.fc2_b = add_vec(m, p + "fc2.b", c.vit_dim);
    m->vit.push_back(L);
  }
  m->post_g = add_vec(m, "vit.post.g", c.vit_dim, 1.0);
  m->post_b = add_vec(m, "vit.post.b", c.vit_dim);
  m->proj_w = add_mat(m, "proj.w", c.lm_dim, d.kproj);
  m->proj_b = add_vec(m, "proj.b", c.lm_dim);
  m->embed = add_mat(m, "lm.embed", c.vocab, c.lm_dim);
  if (c.state_dim > 0) {
    m->state_w = add_mat(m, "state.w", c.lm_dim, c.state_dim);
    m->state_b = add_vec(m, "state.b", c.lm_dim);
  }
  auto dec = [&](const std::string& pre, int layers, int dim, int mlp, bool lm, std::vector<DecLayer>& out) {
    for (int l = 0; l < layers; ++l) {
      const std::string p = pre + std::to_string(l) + ".";
      DecLayer L{-1, -1, -1, -1, -1, -1};
      L.rms1 = add_vec(m, p + "rms1.g", dim, 1.0);
      L.qkv = add_tensor(m, d.qkv_n, dim, m->dt, false, !lm);
      add_param(m, p + "q.w", d.qd, dim, 0.0, L.qkv, MAP_ROPE, 0, c.head_dim);
      add_param(m, p + "k.w", d.kvd, dim, 0.0, L.qkv, MAP_ROPE, d.qd, c.head_dim);
      add_param(m, p + "v.w", d.kvd, dim, 0.0, L.qkv, MAP_IDENT, d.qd + d.kvd);
      if (lm && l == layers - 1 && c.head == VLA_HEAD_PI0) {  // the last LM layer only feeds the cache
        out.push_back(L);
        break;
      }
      L.o = add_mat(m, p + "o.w", dim, d.qd, !lm);
      L.rms2 = add_vec(m, p + "rms2.g", dim, 1.0);
      L.gu = add_tensor(m, 2 * mlp, dim, m->dt, false, !lm);
      add_param(m, p + "gate.w", mlp, dim, 0.0, L.gu, MAP_GATE);
      add_param(m, p + "up.w", mlp, dim, 0.0, L.gu, MAP_UP);
      L.down = add_mat(m, p + "down.w", dim, mlp, !lm);
      out.push_back(L);
    }
  };
  dec("lm.", c.lm_layers, c.lm_dim, c.lm_mlp, true, m->lm);
  if (c.head == VLA_HEAD_DIT) {
    const int de = c.ex_dim;
    m->lm_fin_g = add_vec(m, "lm.final.g", c.lm_dim, 1.0);
    m->in_w = add_mat(m, "ex.in.w", de, c.action_dim, true);
    m->in_b = add_vec(m, "ex.in.b", de);
    m->t1_w = add_mat(m, "ex.time1.w", de, DIT_TIME_DIM, true);
    m->t1_b = add_vec(m, "ex.time1.b", de);
    m->t2_w = add_mat(m, "ex.time2.w", de, de, true);
    m->t2_b = add_vec(m, "ex.time2.b", de);
    for (int l = 0; l < c.ex_layers; ++l) {
      const std::string p = "ex." + std::to_string(l) + ".";
      DitLayer L;
      L.ada_w = add_mat(m, p + "ada.w", 6 * de, de, true);
      L.ada_b = add_vec(m, p + "ada.b", 6 * de);
      if (l % 2 == 0) {  // cross-attention: K / V from the features (M = prefix rows)
        L.q = add_mat(m, p + "q.w", de, de, true);
        L.kv = add_tensor(m, 2 * de, rnd_up(c.lm_dim, 8), m->dt);
        add_param(m, p + "k.w", de, c.lm_dim, 0.0, L.kv, MAP_IDENT, 0);
        add_param(m, p + "v.w", de, c.lm_dim, 0.0, L.kv, MAP_IDENT, de);
      } else {
        L.qkv = add_tensor(m, 3 * de, de, m->dt, false, true);
        add_param(m, p + "q.w", de, de, 0.0, L.qkv, MAP_IDENT, 0);
        add_param(m, p + "k.w", de, de, 0.0, L.qkv, MAP_IDENT, de);
        add_param(m, p + "v.w", de, de, 0.0, L.qkv, MAP_IDENT, 2 * de);
      }
      L.o = add_mat(m, p + "o.w", de, de, true);
      L.fc1 = add_mat(m, p + "fc1.w", c.ex_mlp, de, true);
      L.fc2 = add_mat(m, p + "fc2.w", de, c.ex_mlp, true);
      m->dit.push_back(L);
    }
    m->fada_w = add_mat(m, "ex.final.ada.w", 2 * de, de, true);
    m->fada_b = add_vec(m, "ex.final.ada.b", 2 * de);
    m->out_w = add_mat(m, "ex.out.w", c.action_dim, de, true);
    m->out_b = add_vec(m, "ex.out.b", c.action_dim);
    return;
  }
  if (c.head == VLA_HEAD_COG) {
    const int de = c.ex_dim;
    m->lm_fin_g = add_vec(m, "lm.final.g", c.lm_dim, 1.0);
    m->cog_tok = add_tensor(m, 1, c.lm_dim, DT_F32, true);
    add_param(m, "lm.cog", 1, c.lm_dim, 0.0, m->cog_tok);
    m->cog_w = add_mat(m, "cog.w", de, c.lm_dim);
    m->cog_b = add_vec(m, "cog.b", de);
    m->in_w = add_mat(m, "ex.in.w", de, c.action_dim, true);
    m->in_b = add_vec(m, "ex.in.b", de);
    m->t1_w = add_mat(m, "ex.time1.w", de, DIT_TIME_DIM, true);
    m->t1_b = add_vec(m, "ex.time1.b", de);
    m->t2_w = add_mat(m, "ex.time2.w", de, de, true);
    m->t2_b = add_vec(m, "ex.time2.b", de);
    for (int l = 0; l < c.ex_layers; ++l) {
      const std::string p = "ex." + std::to_string(l) + ".";
      CogLayer L;
      L.ln1_g = add_vec(m, p + "ln1.g", de, 1.0);
      L.ln1_b = add_vec(m, p + "ln1.b", de);
      L.qkv = add_tensor(m, 3 * de, de, m->dt, false, true);
      add_param(m, p + "q.w", de, de, 0.0, L.qkv, MAP_IDENT, 0);
      add_param(m, p + "k.w", de, de, 0.0, L.qkv, MAP_IDENT, de);
      add_param(m, p + "v.w", de, de, 0.0, L.qkv, MAP_IDENT, 2 * de);
      L.o = add_mat(m, p + "o.w", de, de, true);
      L.ln2_g = add_vec(m, p + "ln2.g", de, 1.0);
      L.ln2_b = add_vec(m, p + "ln2.b", de);
      L.fc1 = add_mat(m, p + "fc1.w", c.ex_mlp, de, true);
      L.fc2 = add_mat(m, p + "fc2.w", de, c.ex_mlp, true);
      m->cogl.push_back(L);
    }
    m->fin_g = add_vec(m, "ex.final.g", de, 1.0);
    m->fin_b = add_vec(m, "ex.final.b", de);
    m->out_w = add_mat(m, "ex.out.w", c.action_dim, de, true);
    m->out_b = add_vec(m, "ex.out.b", c.action_dim);
    return;
  }
  m->in_w = add_mat(m, "ex.in.w", c.ex_dim, c.action_dim, true);
  m->in_b = add_vec(m, "ex.in.b", c.ex_dim);
  m->t1_w = add_mat(m, "ex.time1.w", c.ex_dim, 2 * c.ex_dim, true);
  m->t1_b = add_vec(m, "ex.time1.b", c.ex_dim);
  m->t2_w = add_mat(m, "ex.time2.w", c.ex_dim, c.ex_dim, true);
  m->t2_b = add_vec(m, "ex.time2.b", c.ex_dim);
  dec("ex.", c.ex_layers, c.ex_dim, c.ex_mlp, false, m->ex);
  m->fin_g = add_vec(m, "ex.final.g", c.ex_dim, 1.0);
  m->out_w = add_mat(m, "ex.out.w", c.action_dim, c.ex_dim, true);
  m->out_b = add_vec(m, "ex.out.b", c.action_dim);
}

// Generate every parameter of one device tensor into a host image and upload.
static int upload_tensor(vla_model* m, int t, const std::vector<int>& params) {
  const DevTensor& dt = m->T[t];
  std::vector<uint8_t> img(dt.bytes(), 0);
  std::vector<float> vals;
  for (int pi : params) {
    const ParamRec& p = m->P[pi];
    const size_t n = (size_t)p.rows * p.cols;
    vals.resize(n);
    gen_normal(m->seed, p.name.c_str(), n, p.mean, p.stdv, vals.data());
    const bool vec = dt.vec;
    for (int r = 0; r < p.rows; ++r) {
      const int pr = vec ? 0 : dev_row(p, r);
      for (int col = 0; col < p.cols; ++col) {
        const size_t at = vec ? (size_t)p.row_off + col : dt.index(pr, col);
        float v = vals[(size_t)r * p.cols + col];
        if (m->dt == DT_BF16) v = bf16_value(bf16_bits(v));  // the model stores bf16 values
        if (dt.dt == DT_BF16)
          ((uint16_t*)img.data())[at] = bf16_bits(v);
        else
          ((float*)img.data())[at] = v;
      }
    }
  }
  HIP_TRY(hipMemcpy(m->tptr(t), img.data(), img.size(), hipMemcpyHostToDevice));
  return VLA_OK;
}

static int dmalloc(vla_model* m, void** p, size_t bytes) {
  bytes = std::max<size_t>(bytes, 256);
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) return fail(VLA_ENOMEM, std::string("hipMalloc: ") + hipGetErrorString(e));
  m->allocs.push_back(*p);
  return VLA_OK;
}

// ---------------------------------------------------------------------------
// Phase bodies
// ---------------------------------------------------------------------------

struct Run {
  vla_model* m;
  hipStream_t st;
  LaunchCaps caps;
  const Scratch* scr;
  ActWs* aw = nullptr;  // action phase only
  VlmWs* vw = nullptr;  // VLM phase only
};

// Kernel timer: a launch whose tag matches gets a pair of events that its
// main kernel records at its own start and end.
static int timer_events(const Run& r, const char* tag, LaunchCaps* caps) {
  vla_model* m = r.m;
  if (m->timer_tag.empty() || m->timer_tag != tag) return VLA_OK;
  while (m->timer_ev.size() < m->timer_used + 2) {
    hipEvent_t e;
    HIP_TRY(hipEventCreate(&e));
    m->timer_ev.push_back(e);
  }
  caps->ev_start = m->timer_ev[m->timer_used];
  caps->ev_stop = m->timer_ev[m->timer_used + 1];
  m->timer_used += 2;
  return VLA_OK;
}

// Frames of a batched action phase: `n` frames of M rows; the A operand's
// per-frame blocks are a_blk elements apart.
struct Frames {
  int n = 1;
  size_t a_blk = 0;
  int plan_m = 0;  // rows of one frame when M stacks several frames (0: M)
  int plan_batch = 1;  // the most frames a launch of this plan stacks
};

// C = A W[:, koff : koff + K]^T with the epilogue e; W is a weight tensor id.
static GemmDesc gemm_desc(vla_model* m, const void* A, int lda, int W, int M, int N, int K,
                          const Epi& e, int koff = 0, Frames fr = Frames()) {
  const DevTensor& t = m->T[W];
  GemmDesc g{m->dt, A, lda, m->tptr(W), t.ld, M, N, K, e};
  if (t.fks > 0) {
    g.frag_ks = t.fks;
    g.frag_ks0 = koff / frag_slab(m->dt);
  } else {
    g.W = m->tptr(W) + (size_t)koff * m->esz;
  }
  g.frames = fr.n;
  g.a_blk = fr.a_blk;
  g.plan_m = fr.plan_m;
  g.plan_batch = fr.plan_batch;
  return g;
}

static int gemm(const Run& r, const char* tag, const void* A, int lda, int W, int M, int N, int K,
                const Epi& e, int koff = 0, Frames fr = Frames()) {
  vla_model* m = r.m;
  const GemmDesc g = gemm_desc(m, A, lda, W, M, N, K, e, koff, fr);
  LaunchCaps caps = r.caps;
  VLA_TRY(timer_events(r, tag, &caps));
  hipError_t err = launch_gemm(g, *r.scr, caps, r.st);
  if (err != hipSuccess)
    return fail(VLA_EHIP, std::string("gemm ") + std::to_string(M) + "x" + std::to_string(N) + "x" +
                              std::to_string(K) + ": " + hipGetErrorString(err));
  return VLA_OK;
}

// C = A W^T with W a row-major [N][ldw] matrix in device memory (not a model
// tensor id): the batched action loop's row-major expert weights.
static int gemm_rm(const Run& r, const char* tag, const void* A, int lda, const void* W, int ldw, int M, int N,
                   int K, const Epi& e, Frames fr = Frames()) {
  vla_model* m = r.m;
  GemmDesc g{m->dt, A, lda, W, ldw, M, N, K, e};
  g.plan_m = fr.plan_m;
  g.plan_batch = fr.plan_batch;
  LaunchCaps caps = r.caps;
  VLA_TRY(timer_events(r, tag, &caps));
  hipError_t err = launch_gemm(g, *r.scr, caps, r.st);
  if (err != hipSuccess)
    return fail(VLA_EHIP, std::string("gemm ") + std::to_string(M) + "x" + std::to_string(N) + "x" +
                              std::to_string(K) + ": " + hipGetErrorString(err));
  return VLA_OK;
}

static int attn_kv(const Run& r, const char* tag, const AttnKvDesc& a0) {
  LaunchCaps caps = r.caps;
  VLA_TRY(timer_events(r, tag, &caps));
  AttnKvDesc a = a0;
  if (r.aw) {  // action phases: the lane's room for key splits
    a.part = r.aw->apart;
    a.part_floats = r.aw->apart_floats;
    a.cnt = r.aw->acnt;
    a.cnt_n = r.aw->acnt_n;
  }
  hipError_t err = launch_attention_kv(a, caps, r.st);
  if (err != hipSuccess) return fail(VLA_EHIP, std::string("attention: ") + hipGetErrorString(err));
  return VLA_OK;
}

static int attn(const Run& r, const char* tag, const AttnDesc& a) {
  LaunchCaps caps = r.caps;
  VLA_TRY(timer_events(r, tag, &caps));
  hipError_t err = launch_attention(a, *r.scr, caps, r.st);
  if (err != hipSuccess) return fail(VLA_EHIP, std::string("attention: ") + hipGetErrorString(err));
  return VLA_OK;
}

// Residual add of `splits` pending partials (from the phase scratch) + bias,
// then LayerNorm / RMSNorm into `out`.
static int run_norm(const Run& r, NormDesc n) {
  n.dtype = r.m->dt;
  n.part = r.scr->ptr;
  hipError_t err = launch_norm(n, r.st);
  if (err != hipSuccess) return fail(VLA_EHIP, std::string("norm: ") + hipGetErrorString(err));
  return VLA_OK;
}

// out: row-major [rows][d], or the row-block operand layout when it feeds a
// skinny GEMM (afrag)
static int norm(const Run& r, float* x, int rows, int d, int splits, const float* bias, int g, int b,
                bool rms, void* out, bool afrag = false, int blk_rows = 0, size_t blk_out = 0) {
  NormDesc n;
  n.blk_rows = blk_rows;
  n.blk_out = blk_out;
  n.x = x;
  n.ldx = d;
  n.rows = rows;
  n.d = d;
  n.splits = splits;
  n.bias = bias;
  n.g = r.m->f32(g);
  n.b = b >= 0 ? r.m->f32(b) : nullptr;
  n.rms = rms;
  n.out = out;
  n.ldo = d;
  n.afrag = afrag;
  return run_norm(r, n);
}

// GEMM whose result is added to the residual stream by the next norm: the raw
// result (or its split-K partials) goes to the phase scratch.
static int gemm_part_rm(const Run& r, const char* tag, const void* A, int lda, const void* W, int ldw, int M,
                        int N, int K, int* splits, Frames fr) {
  vla_model* m = r.m;
  Epi e;
  e.kind = EPI_PART;
  e.out = r.scr->ptr;
  e.ldo = (int)std::min<size_t>(r.scr->floats, (size_t)INT32_MAX);
  GemmDesc g{m->dt, A, lda, W, ldw, M, N, K, e};
  g.plan_m = fr.plan_m;
  g.plan_batch = fr.plan_batch;
  *splits = plan_gemm(g).splits;
  return gemm_rm(r, tag, A, lda, W, ldw, M, N, K, e, fr);
}

static int gemm_part(const Run& r, const char* tag, const void* A, int lda, int W, int M, int N,
                     int K, int* splits, Frames fr = Frames()) {
  vla_model* m = r.m;
  Epi e;
  e.kind = EPI_PART;
  e.out = r.scr->ptr;
  e.ldo = (int)std::min<size_t>(r.scr->floats, (size_t)INT32_MAX);
  if (fr.n > 1) e.blk_rows = M;
  *splits = plan_gemm(gemm_desc(m, A, lda, W, M, N, K, e, 0, fr)).splits;
  return gemm(r, tag, A, lda, W, M, N, K, e, 0, fr);
}

// Split-K skinny GEMM whose partials the kernel itself adds to the residual
// x, leaving h = x * gain (row-block operand layout) and the rows' sums of
// squares for the next GEMM: an RMSNorm folded across two launches (see
// Epi::rowss). One frame.
static int gemm_part_fold(const Run& r, const char* tag, const void* A, int lda, int W, int M, int N, int K,
                          float* x, int g, void* h) {
  Epi e;
  e.kind = EPI_PART;
  e.out = r.scr->ptr;
  e.ldo = (int)std::min<size_t>(r.scr->floats, (size_t)INT32_MAX);
  e.x = x;
  e.ldx = N;
  e.norm_g = r.m->f32(g);
  e.norm_out = h;
  e.afrag = 1;
  e.rowss = r.aw->rowss;
  e.cnt = r.aw->pcnt;
  return gemm(r, tag, A, lda, W, M, N, K, e, 0, Frames());
}

// the consumer side: scale each row of the product by the folded norm's 1/rms
static void fold_consumer(const Run& r, Epi& e, int d) {
  e.rowss = r.aw->rowss;
  e.rowss_n = (d + 31) / 32;
  e.rowss_d = d;
}

static Epi epi_kind(int kind, void* out = nullptr, int ldo = 0, const float* bias = nullptr) {
  Epi e;
  e.kind = kind;
  e.out = out;
  e.ldo = ldo;
  e.bias = bias;
  return e;
}

// One Gemma-style decoder layer: RMSNorm (after adding the pending residual
// partials) -> QKV (+RoPE, K/V stored) -> attention over [past; own] -> O ->
// RMSNorm (after adding O) -> GeGLU -> down. The down projection is left
// pending in the scratch (*pend = its split count) for the next norm. In a
// one-frame expert layer both norms are folded into the GEMMs around them
// (gemm_part_fold, fold_consumer): the O projection leaves h = x * rms2 for
// the gate/up GEMM, and the down projection x * next_g (the next norm's
// gain) with *pend = -1, so the layer is five launches.
// Several frames may run together, `rows` rows each:
//  * LM layers (a batched prefill): x holds the frames' rows one after
//    another, frame f's own K/V (its cache) sit kstride / vstride elements
//    after frame f - 1's;
//  * expert layers of a batched action loop, wide (wl set): the same
//    stacked rows and row-major operands, the tiled GEMM over all frames'
//    rows with the row-major copies of the layer's matrices in *wl;
//  * otherwise expert layers take frame blocks in the row-block operand
//    layout (skinny GEMMs, one launch for all frames).
// Frame f of a batched expert layer reads the past K/V kpast[f] / vpast[f]
// and the action workspace's per-frame blocks. Stacked rows get split-K
// factors planned for a fixed row count (one frame's prefix in the LM, the
// largest batched loop in the expert), so a frame's result does not depend
// on how many frames share the launch.
static int decoder_layer(const Run& r, bool lm, const DecLayer& L, float* x, int rows, int dim, int mlp,
                         void* h, void* q, void* kout, void* vout, int pos0, const void* const* kpast,
                         const void* const* vpast, int npast, void* att, void* mlpbuf, bool kv_only,
                         int* pend, int frames = 1, size_t kstride = 0, size_t vstride = 0,
                         const vla_model::WideLayer* wl = nullptr, int next_g = -1) {
  vla_model* m = r.m;
  const vla_config& c = m->c;
  const Dims& d = m->d;
  const bool wide = !lm && wl;
  const bool stacked = lm || wide;  // row-major operands, frames' rows stacked into M
  const bool af = !stacked;         // skinny operands: row-block operand layout
  const bool fb = frames > 1;       // frame blocks
  const ActWs* aw = r.aw;
  if (!lm && fb && !aw) return fail(VLA_EINVAL, "batched frames: expert layers need an action workspace");
  if (lm && fb && (kstride == 0 || vstride == 0)) return fail(VLA_EINVAL, "batched prefill: cache strides");
  const int gm = stacked ? frames * rows : rows;
  auto frm = [&](size_t a_blk) {
    Frames f;
    if (stacked) {
      // splits: those of one frame's prefix rows (LM; planned for prefill
      // batches of up to MAX_VLM_BATCH frames), or of the largest batched
      // action loop (expert): fixed for every group size
      f.plan_m = lm ? rows : MAX_ACT_BATCH * rows;
      if (lm) f.plan_batch = MAX_VLM_BATCH;
    } else {
      f.n = frames;
      f.a_blk = fb ? a_blk : 0;
    }
    return f;
  };
  const bool skin_fb = fb && !stacked;  // skinny frame blocks
  const int nblk = skin_fb ? rows : 0;   // norm output frame blocks (operand layout)
  const size_t nblk_out = skin_fb ? aw->blk_de : 0;
  const bool fold = !lm && af && !fb && aw && aw->rowss;
  const bool folded_in = *pend < 0;  // h holds x * rms1 already
  if (folded_in && !fold) return fail(VLA_ESTATE, "a folded norm is pending outside a one-frame expert layer");
  if (!folded_in) VLA_TRY(norm(r, x, frames * rows, dim, *pend, nullptr, L.rms1, -1, true, h, af, nblk, nblk_out));
  *pend = 0;
  Epi e;
  e.kind = EPI_QKV_ROPE;
  e.q = q;
  e.ldq = d.qd;
  e.k = kout;
  e.v = vout;
  e.kv_nb = (lm ? d.prefix_pad : d.chunk_pad) / 32;
  e.nq = c.lm_heads;
  e.nkv = c.lm_kv_heads;
  e.hd = c.head_dim;
  e.pos0 = pos0;
  e.rope_cos = m->rope_cos;
  e.rope_sin = m->rope_sin;
  if (fb) {
    e.blk_rows = rows;
    e.blk_k = lm ? kstride : aw->blk_k;
    e.blk_v = lm ? vstride : aw->blk_v;
  }
  if (folded_in) fold_consumer(r, e, dim);
  const char* tq = lm ? "lm.qkv" : "ex.qkv";
  if (wide)
    VLA_TRY(gemm_rm(r, tq, h, dim, wl->qkv, dim, gm, d.qkv_n, dim, e, frm(0)));
  else
    VLA_TRY(gemm(r, tq, h, dim, L.qkv, gm, d.qkv_n, dim, e, 0, frm(skin_fb ? aw->blk_de : 0)));
  if (kv_only) return VLA_OK;
  AttnKvDesc a{};
  a.dtype = m->dt;
  a.q = q;
  a.ldq = d.qd;
  if (kpast) {
    a.k0 = kpast[0];
    a.v0 = vpast[0];
    a.S0 = npast;
    a.k1 = kout;
    a.v1 = vout;
    a.S1 = rows;
  } else {
    a.k0 = kout;
    a.v0 = vout;
    a.S0 = rows;
  }
  a.out = att;
  a.ldo = d.qd;
  a.out_afrag = af;
  a.Sq = rows;
  a.nq = c.lm_heads;
  a.nkv = c.lm_kv_heads;
  a.hd = c.head_dim;
  if (fb && lm) {
    // frame f: queries f * rows .., its own cache, output rows f * rows ..
    a.frames = frames;
    for (int f = 1; f < frames; ++f) {
      a.k0f[f] = (const char*)kout + f * kstride * m->esz;
      a.v0f[f] = (const char*)vout + f * vstride * m->esz;
    }
    a.out_blk = (size_t)rows * d.qd;
  } else if (fb) {
    if (!kpast) return fail(VLA_EINVAL, "batched frames need past K/V");
    a.frames = frames;
    for (int f = 1; f < frames; ++f) {
      a.k0f[f] = kpast[f];
      a.v0f[f] = vpast[f];
    }
    a.k1_blk = aw->blk_k;
    a.v1_blk = aw->blk_v;
    a.out_blk = wide ? (size_t)rows * d.qd : aw->blk_att;
  }
  VLA_TRY(attn_kv(r, lm ? "lm.attn" : "ex.attn", a));
  int so = 0;
  const char* to = lm ? "lm.o" : "ex.o";
  if (fold) {
    VLA_TRY(gemm_part_fold(r, to, att, d.qd, L.o, gm, dim, d.qd, x, L.rms2, h));
  } else {
    if (wide)
      VLA_TRY(gemm_part_rm(r, to, att, d.qd, wl->o, d.qd, gm, dim, d.qd, &so, frm(0)));
    else
      VLA_TRY(gemm_part(r, to, att, d.qd, L.o, gm, dim, d.qd, &so, frm(skin_fb ? aw->blk_att : 0)));
    VLA_TRY(norm(r, x, frames * rows, dim, so, nullptr, L.rms2, -1, true, h, af, nblk, nblk_out));
  }
  Epi eg = epi_kind(EPI_GEGLU, mlpbuf, mlp);
  eg.afrag = af;
  if (fold) fold_consumer(r, eg, dim);
  if (skin_fb) {
    eg.blk_rows = rows;
    eg.blk_out = aw->blk_mlp;
  }
  const char* tg = lm ? "lm.gateup" : "ex.gateup";
  if (wide)
    VLA_TRY(gemm_rm(r, tg, h, dim, wl->gu, dim, gm, 2 * mlp, dim, eg, frm(0)));
  else
    VLA_TRY(gemm(r, tg, h, dim, L.gu, gm, 2 * mlp, dim, eg, 0, frm(skin_fb ? aw->blk_de : 0)));
  const char* td = lm ? "lm.down" : "ex.down";
  if (fold && next_g >= 0) {
    VLA_TRY(gemm_part_fold(r, td, mlpbuf, mlp, L.down, gm, dim, mlp, x, next_g, h));
    *pend = -1;
  } else if (wide) {
    VLA_TRY(gemm_part_rm(r, td, mlpbuf, mlp, wl->down, mlp, gm, dim, mlp, pend, frm(0)));
  } else {
    VLA_TRY(gemm_part(r, td, mlpbuf, mlp, L.down, gm, dim, mlp, pend, frm(skin_fb ? aw->blk_mlp : 0)));
  }
  return VLA_OK;
}

// The VLM prefill of `n` frames together (a batched prefill; n <= the lane's
// capacity): their views are stacked as n * n_views views for the ViT and
// their prefixes as n * prefix rows for the LM, each frame writing its own
// context ctxs[f] (consecutive contexts of one block when n > 1). Splits
// and reductions are planned for one frame, so every frame's cache equals
// its own prefill bit for bit.
static int run_prefill_n(const Run& r, const vla_frame* f, int n, vla_ctx* const* ctxs) {
  vla_model* m = r.m;
  const vla_config& c = m->c;
  const Dims& d = m->d;
  VlmWs& w = *r.vw;
  if (n < 1 || n > w.cap) return fail(VLA_EINVAL, "frames per prefill exceed the lane's capacity");
  if (n > 1 && !ctx_consecutive(m, ctxs, n)) return fail(VLA_EINVAL, "batched prefill: contexts not consecutive");
  const int dv = c.vit_dim, dl = c.lm_dim, rows = d.rows_v, P = d.prefix;
  const int nv = n * c.n_views;  // views of all frames
  auto fr1 = [&](int rows1) {  // splits of one frame's rows, for prefill batches
    Frames x;
    x.plan_m = rows1;
    x.plan_batch = MAX_VLM_BATCH;
    return x;
  };
  // ViT: patch embedding + bias + position
  for (int i = 0; i < n; ++i)
    HIP_TRY(launch_patchify(m->dt, f[i].pixels, c.n_views, c.img_h, c.img_w, c.patch,
                            (char*)w.h + (size_t)i * rows * d.kp_pad * m->esz, d.kp_pad, r.st));
  {
    Epi e = epi_kind(EPI_F32, w.xv, dv, m->f32(m->patch_b));
    e.rowadd = m->f32(m->pos);
    e.rowadd_period = d.tview;
    e.ldra = dv;
    VLA_TRY(gemm(r, "vit.patch", w.h, d.kp_pad, m->patch_w, n * rows, dv, d.kp_pad, e, 0, fr1(rows)));
  }
  int pend = 0;
  const float* pbias = nullptr;
  for (int l = 0; l < c.vit_layers; ++l) {
    const VitLayer& L = m->vit[l];
    VLA_TRY(norm(r, w.xv, n * rows, dv, pend, pbias, L.ln1_g, L.ln1_b, false, w.h));
    VLA_TRY(gemm(r, "vit.qkv", w.h, dv, L.qkv_w, n * rows, 3 * dv, dv,
                 epi_kind(EPI_T, w.qkv, 3 * dv, m->f32(L.qkv_b)), 0, fr1(rows)));
    AttnDesc a{};
    a.dtype = m->dt;
    a.q = w.qkv;
    a.ldq = 3 * dv;
    a.k0 = (char*)w.qkv + dv * m->esz;
    a.v0 = (char*)w.qkv + 2 * dv * m->esz;
    a.S0 = d.tview;
    a.ldkv = 3 * dv;
    a.out = w.att;
    a.ldo = dv;
    a.Sq = d.tview;
    a.nq = a.nkv = c.vit_heads;
    a.hd = d.vhd;
    a.segs = nv;
    a.plan_segs = c.n_views;
    a.seg_q = a.seg_kv = (long long)d.tview * 3 * dv;
    a.seg_o = (long long)d.tview * dv;
    VLA_TRY(attn(r, "vit.attn", a));
    int so = 0;
    VLA_TRY(gemm_part(r, "vit.o", w.att, dv, L.o_w, n * rows, dv, dv, &so, fr1(rows)));
    VLA_TRY(norm(r, w.xv, n * rows, dv, so, m->f32(L.o_b), L.ln2_g, L.ln2_b, false, w.h));
    VLA_TRY(gemm(r, "vit.fc1", w.h, dv, L.fc1_w, n * rows, c.vit_mlp, dv,
                 epi_kind(EPI_GELU, w.mlp, c.vit_mlp, m->f32(L.fc1_b)), 0, fr1(rows)));
    VLA_TRY(gemm_part(r, "vit.fc2", w.mlp, c.vit_mlp, L.fc2_w, n * rows, dv, c.vit_mlp, &pend, fr1(rows)));
    pbias = m->f32(L.fc2_b);
  }
  {
    // final LayerNorm; the pixel shuffle (if any) is the norm's output placement
    NormDesc nd;
    nd.x = w.xv;
    nd.ldx = dv;
    nd.rows = n * rows;
    nd.d = dv;
    nd.splits = pend;
    nd.bias = pbias;
    nd.g = m->f32(m->post_g);
    nd.b = m->f32(m->post_b);
    nd.out = w.h;
    nd.ldo = d.kproj;
    nd.shuffle = c.shuffle;
    nd.grid_w = d.gw;
    nd.tview = d.tview;
    VLA_TRY(run_norm(r, nd));
  }
  // prefix of frame i at rows i * P: [projected image tokens; text * sqrt(d);
  // state projection]
  for (int i = 0; i < n; ++i) {
    float* xl = w.xl + (size_t)i * P * dl;
    VLA_TRY(gemm(r, "proj", (char*)w.h + (size_t)i * d.nimg * d.kproj * m->esz, d.kproj, m->proj_w, d.nimg,
                 dl, d.kproj, epi_kind(EPI_F32, xl, dl, m->f32(m->proj_b))));
    HIP_TRY(launch_embed(m->dt, m->tptr(m->embed), dl, c.vocab, f[i].text_ids, c.n_text, std::sqrt((float)dl),
                         xl + (size_t)d.nimg * dl, dl, r.st));
    if (c.head == VLA_HEAD_COG)  // the learned cognition token, the prefix's last row
      HIP_TRY(launch_copy(xl + (size_t)(P - 1) * dl, m->f32(m->cog_tok), (size_t)dl * 4, r.st));
    if (c.state_dim > 0) {
      void* sb = (char*)w.sbuf + (size_t)i * d.s_pad * m->esz;
      HIP_TRY(launch_cvt_pad(m->dt, f[i].state, 1, c.state_dim, sb, d.s_pad, false, nullptr, r.st));
      VLA_TRY(gemm(r, "state", sb, d.s_pad, m->state_w, 1, dl, d.s_pad,
                   epi_kind(EPI_F32, xl + (size_t)(P - 1) * dl, dl, m->f32(m->state_b))));
    }
  }
  // LM prefill writing the caches
  const size_t layer_k = ctx_layer_k(m) * m->esz;
  const size_t layer_v = ctx_layer_v(m) * m->esz;
  const size_t kstride = ctx_kbytes(m) / m->esz, vstride = ctx_vbytes(m) / m->esz;
  pend = 0;
  const bool dit = c.head == VLA_HEAD_DIT;
  vla_ctx* ctx = ctxs[0];
  for (int l = 0; l < c.lm_layers; ++l) {
    void* K = (char*)ctx->K + l * layer_k;
    void* V = (char*)ctx->V + l * layer_v;
    VLA_TRY(decoder_layer(r, true, m->lm[l], w.xl, P, dl, c.lm_mlp, w.h, w.qkv, K, V, 0, nullptr, nullptr, 0,
                          w.att, w.mlp, c.head == VLA_HEAD_PI0 && l == c.lm_layers - 1, &pend, n, kstride,
                          vstride));
  }
  if (c.head == VLA_HEAD_COG) {
    // features = final RMSNorm of the last layer; the hand-off is the
    // cognition row's projection c = W_c f + b_c, one per frame
    VLA_TRY(norm(r, w.xl, n * P, dl, pend, nullptr, m->lm_fin_g, -1, true, w.h));
    for (int i = 0; i < n; ++i)
      VLA_TRY(gemm(r, "cog", (char*)w.h + ((size_t)i * P + P - 1) * dl * m->esz, dl, m->cog_w, 1, c.ex_dim, dl,
                   epi_kind(EPI_F32, ctxs[i]->cog, c.ex_dim, m->f32(m->cog_b))));
  }
  if (dit) {
    // features = final RMSNorm of the last layer; then the cross K/V of every
    // even DiT layer, once per frame
    VLA_TRY(norm(r, w.xl, n * P, dl, pend, nullptr, m->lm_fin_g, -1, true, w.h));
    const size_t xe = cross_elems(m) * m->esz;
    for (int l = 0; l < c.ex_layers; l += 2) {
      Epi e;
      e.kind = EPI_QKV_PLAIN;
      e.nq = 0;
      e.nkv = c.ex_heads;
      e.hd = d.ehd;
      e.k = (char*)ctx->XK + (l / 2) * xe;
      e.v = (char*)ctx->XV + (l / 2) * xe;
      e.kv_nb = d.prefix_pad / 32;
      if (n > 1) {
        e.blk_rows = P;
        e.blk_k = e.blk_v = ctx_xbytes(m) / m->esz;
      }
      VLA_TRY(gemm(r, "dit.cross_kv", w.h, dl, m->dit[l].kv, n * P, 2 * c.ex_dim, dl, e, 0, fr1(P)));
    }
  }
  return VLA_OK;
}

static int run_prefill(const Run& r, const vla_frame* f, vla_ctx* ctx) { return run_prefill_n(r, f, 1, &ctx); }

// GR00T-style DiT head (Euler steps as in run_denoise): tokens = W_a x + b_a +
// positions; per layer, adaLN-modulated LayerNorm (gain 1 + scale, shift
// from the per-step table) -> attention (even layers: queries over the
// frame's cross K/V; odd layers: self-attention) -> out-projection whose
// partial sums the next norm adds with gate1 -> adaLN LayerNorm -> GELU MLP
// -> down-projection added with gate2 by the next norm; final adaLN +
// out-projection fused with the Euler update.
static int run_denoise_dit(const Run& r, const vla_ctx* ctx, const float* noise, float* x) {
  vla_model* m = r.m;
  const vla_config& c = m->c;
  const Dims& d = m->d;
  ActWs& w = *r.aw;
  const int H = c.chunk_len, de = c.ex_dim, A = c.action_dim, L = c.ex_layers;
  const size_t xe = cross_elems(m) * m->esz;
  HIP_TRY(launch_cvt_pad(m->dt, noise, H, A, w.xop, d.a_pad, true, x, r.st));
  auto adanorm = [&](int pend, const float* gate, const float* shift, const float* scale) {
    NormDesc n;
    n.x = w.u;
    n.ldx = de;
    n.rows = H;
    n.d = de;
    n.splits = pend;
    n.colscale = gate;
    n.g = scale;
    n.g_plus_one = 1;
    n.b = shift;
    n.out = w.h;
    n.ldo = de;
    n.afrag = 1;
    return run_norm(r, n);
  };
  for (int k = 0; k < c.n_steps; ++k) {
    {
      Epi e = epi_kind(EPI_F32, w.u, de, m->f32(m->in_b));
      e.rowadd = m->dpos;
      e.rowadd_period = H;
      e.ldra = de;
      VLA_TRY(gemm(r, "ex.in", w.xop, d.a_pad, m->in_w, H, de, d.a_pad, e));
    }
    int pend = 0;
    const float* pgate = nullptr;
    for (int l = 0; l < L; ++l) {
      const DitLayer& D = m->dit[l];
      const float* ad = m->ada + ((size_t)k * L + l) * 6 * de;
      VLA_TRY(adanorm(pend, pgate, ad, ad + de));
      AttnKvDesc a{};
      a.dtype = m->dt;
      a.q = w.q;
      a.ldq = de;
      a.nq = a.nkv = c.ex_heads;
      a.hd = d.ehd;
      a.Sq = H;
      a.out = w.att;
      a.out_afrag = 1;
      if (l % 2 == 0) {
        VLA_TRY(gemm(r, "ex.q", w.h, de, D.q, H, de, de, epi_kind(EPI_T, w.q, de)));
        a.k0 = (const char*)ctx->XK + (l / 2) * xe;
        a.v0 = (const char*)ctx->XV + (l / 2) * xe;
        a.S0 = d.prefix;
      } else {
        Epi e;
        e.kind = EPI_QKV_PLAIN;
        e.q = w.q;
        e.ldq = de;
        e.nq = c.ex_heads;
        e.nkv = c.ex_heads;
        e.hd = d.ehd;
        e.k = w.kown;
        e.v = w.vown;
        e.kv_nb = d.chunk_pad / 32;
        VLA_TRY(gemm(r, "ex.qkv", w.h, de, D.qkv, H, 3 * de, de, e));
        a.k0 = w.kown;
        a.v0 = w.vown;
        a.S0 = H;
      }
      VLA_TRY(attn_kv(r, "ex.attn", a));
      int so = 0;
      VLA_TRY(gemm_part(r, "ex.o", w.att, de, D.o, H, de, de, &so));
      VLA_TRY(adanorm(so, ad + 2 * de, ad + 3 * de, ad + 4 * de));
      Epi e1 = epi_kind(EPI_GELU, w.mlp, c.ex_mlp);
      e1.afrag = 1;
      VLA_TRY(gemm(r, "ex.fc1", w.h, de, D.fc1, H, c.ex_mlp, de, e1));
      VLA_TRY(gemm_part(r, "ex.fc2", w.mlp, c.ex_mlp, D.fc2, H, de, c.ex_mlp, &pend));
      pgate = ad + 5 * de;
    }
    const float* fa = m->fada + (size_t)k * 2 * de;
    VLA_TRY(adanorm(pend, pgate, fa, fa + de));
    Epi e;
    e.kind = EPI_EULER;
    e.afrag = 1;
    e.bias = m->f32(m->out_b);
    e.x = x;
    e.ldx = A;
    e.xop = w.xop;
    e.ldxop = d.a_pad;
    e.dt = m->step_b[k];
    e.xs = m->step_a[k];
    VLA_TRY(gemm(r, "ex.out", w.h, de, m->out_w, H, A, de, e));
  }
  return VLA_OK;
}

// Cognition-token head (DDIM or Euler steps as in run_denoise): the token
// sequence [action tokens (W_a x + b_a + positions); the frame's cognition
// vector; the step's time token] runs through pre-LN self-attention layers
// (LayerNorm -> fused q|k|v -> attention over all tokens -> out-projection
// whose partial sums the next norm adds -> LayerNorm -> GELU MLP ->
// down-projection added by the next norm); the final LayerNorm's action rows
// feed the out-projection fused with the sampler update.
static int run_denoise_cog(const Run& r, const vla_ctx* ctx, const float* noise, float* x) {
  vla_model* m = r.m;
  const vla_config& c = m->c;
  const Dims& d = m->d;
  ActWs& w = *r.aw;
  const int H = c.chunk_len, de = c.ex_dim, A = c.action_dim, S = d.arows;
  if (!ctx->cog) return fail(VLA_ESTATE, "context has no cognition vector");
  HIP_TRY(launch_cvt_pad(m->dt, noise, H, A, w.xop, d.a_pad, true, x, r.st));
  auto ln = [&](int pend, int g, int b) {
    NormDesc n;
    n.x = w.u;
    n.ldx = de;
    n.rows = S;
    n.d = de;
    n.splits = pend;
    n.g = m->f32(g);
    n.b = m->f32(b);
    n.out = w.h;
    n.ldo = de;
    n.afrag = 1;
    return run_norm(r, n);
  };
  for (int k = 0; k < c.n_steps; ++k) {
    {
      Epi e = epi_kind(EPI_F32, w.u, de, m->f32(m->in_b));
      e.rowadd = m->dpos;
      e.rowadd_period = H;
      e.ldra = de;
      VLA_TRY(gemm(r, "ex.in", w.xop, d.a_pad, m->in_w, H, de, d.a_pad, e));
    }
    HIP_TRY(launch_copy(w.u + (size_t)H * de, ctx->cog, (size_t)de * 4, r.st));
    HIP_TRY(launch_copy(w.u + (size_t)(H + 1) * de, m->ttok + (size_t)k * de, (size_t)de * 4, r.st));
    int pend = 0;
    for (int l = 0; l < c.ex_layers; ++l) {
      const CogLayer& L = m->cogl[l];
      VLA_TRY(ln(pend, L.ln1_g, L.ln1_b));
      Epi e;
      e.kind = EPI_QKV_PLAIN;
      e.q = w.q;
      e.ldq = de;
      e.nq = c.ex_heads;
      e.nkv = c.ex_heads;
      e.hd = d.ehd;
      e.k = w.kown;
      e.v = w.vown;
      e.kv_nb = d.chunk_pad / 32;
      VLA_TRY(gemm(r, "ex.qkv", w.h, de, L.qkv, S, 3 * de, de, e));
      AttnKvDesc a{};
      a.dtype = m->dt;
      a.q = w.q;
      a.ldq = de;
      a.k0 = w.kown;
      a.v0 = w.vown;
      a.S0 = S;
      a.nq = a.nkv = c.ex_heads;
      a.hd = d.ehd;
      a.Sq = S;
      a.out = w.att;
      a.out_afrag = 1;
      VLA_TRY(attn_kv(r, "ex.attn", a));
      int so = 0;
      VLA_TRY(gemm_part(r, "ex.o", w.att, de, L.o, S, de, de, &so));
      VLA_TRY(ln(so, L.ln2_g, L.ln2_b));
      Epi e1 = epi_kind(EPI_GELU, w.mlp, c.ex_mlp);
      e1.afrag = 1;
      VLA_TRY(gemm(r, "ex.fc1", w.h, de, L.fc1, S, c.ex_mlp, de, e1));
      VLA_TRY(gemm_part(r, "ex.fc2", w.mlp, c.ex_mlp, L.fc2, S, de, c.ex_mlp, &pend));
    }
    VLA_TRY(ln(pend, m->fin_g, m->fin_b));
    Epi e;
    e.kind = EPI_EULER;
    e.afrag = 1;
    e.bias = m->f32(m->out_b);
    e.x = x;
    e.ldx = A;
    e.xop = w.xop;
    e.ldxop = d.a_pad;
    e.dt = m->step_b[k];
    e.xs = m->step_a[k];
    VLA_TRY(gemm(r, "ex.out", w.h, de, m->out_w, H, A, de, e));
  }
  return VLA_OK;
}

// Row-major copies of the expert layers' matrices for batched action loops
// (converted on the device from the fragment-ordered weights, once). Not
// while a graph is being captured.
static int ensure_wide(vla_model* m) {
  if (!m->exw.empty()) return VLA_OK;
  const vla_config& c = m->c;
  struct Item {
    int t, N, K;
  };
  std::vector<Item> items;
  for (const DecLayer& L : m->ex) {
    const int de = c.ex_dim;
    items.push_back({L.qkv, m->d.qkv_n, de});
    items.push_back({L.o, de, m->d.qd});
    items.push_back({L.gu, 2 * c.ex_mlp, de});
    items.push_back({L.down, de, c.ex_mlp});
  }
  std::vector<size_t> off;
  size_t total = 0;
  for (const Item& it : items) {
    off.push_back(total);
    total += ((size_t)it.N * it.K * m->esz + 255) / 256 * 256;
  }
  HIP_TRY(hipMalloc(&m->exw_mem, total));
  for (size_t i = 0; i < items.size(); ++i) {
    const Item& it = items[i];
    const DevTensor& t = m->T[it.t];
    if (t.fks <= 0 || t.rows != it.N || t.ld != it.K) return fail(VLA_ESTATE, "expert weight layout");
    HIP_TRY(launch_unfrag(m->dt, m->tptr(it.t), it.N, it.K, t.fks, (char*)m->exw_mem + off[i], nullptr));
  }
  HIP_TRY(hipDeviceSynchronize());
  for (size_t l = 0; l < m->ex.size(); ++l) {
    vla_model::WideLayer w;
    w.qkv = (char*)m->exw_mem + off[4 * l];
    w.o = (char*)m->exw_mem + off[4 * l + 1];
    w.gu = (char*)m->exw_mem + off[4 * l + 2];
    w.down = (char*)m->exw_mem + off[4 * l + 3];
    m->exw.push_back(w);
  }
  return VLA_OK;
}

// The flow-matching loop of `frames` frames together (at most MAX_ACT_BATCH; noise
// and x hold the frames' chunks one after another): the frames' rows share
// every weight load, and each frame's result equals its own run bit for bit.
static int run_denoise_n(const Run& r, const vla_ctx* const* ctxs, int frames, const float* noise, float* x) {
  vla_model* m = r.m;
  if (m->c.head == VLA_HEAD_DIT || m->c.head == VLA_HEAD_COG) {
    if (frames != 1) return fail(VLA_EINVAL, "batched action phases: pi0-style head only");
    return m->c.head == VLA_HEAD_DIT ? run_denoise_dit(r, ctxs[0], noise, x) : run_denoise_cog(r, ctxs[0], noise, x);
  }
  if (frames < 1 || frames > MAX_ACT_BATCH) return fail(VLA_EINVAL, "frames per action phase: 1 to " + std::to_string(MAX_ACT_BATCH));
  if (frames > 1 && m->exw.size() != m->ex.size()) return fail(VLA_ESTATE, "row-major expert weights missing");
  const vla_config& c = m->c;
  const Dims& d = m->d;
  ActWs& w = *r.aw;
  const int H = c.chunk_len, de = c.ex_dim, A = c.action_dim;
  const bool fb = frames > 1;
  const int blk = fb ? H : 0;
  auto frm = [&](size_t a_blk) { Frames f; f.n = frames; f.a_blk = fb ? a_blk : 0; return f; };
  // every operand of the expert's GEMMs is in the row-block operand layout
  HIP_TRY(launch_cvt_pad(m->dt, noise, frames * H, A, w.xop, d.a_pad, true, x, r.st, blk, w.blk_xop));
  const size_t layer_k = ctx_layer_k(m) * m->esz;
  const size_t layer_v = ctx_layer_v(m) * m->esz;
  for (int k = 0; k < c.n_steps; ++k) {
    // action embedding and time conditioning
    Epi ein = epi_kind(EPI_T, w.a, de, m->f32(m->in_b));
    ein.afrag = 1;
    ein.blk_rows = blk;
    ein.blk_out = w.blk_de;
    VLA_TRY(gemm(r, "ex.in", w.xop, d.a_pad, m->in_w, H, de, d.a_pad, ein, 0, frm(w.blk_xop)));
    Epi et1 = epi_kind(EPI_SWISH, w.hid, de, m->ck + (size_t)k * de);
    et1.afrag = 1;
    et1.blk_rows = blk;
    et1.blk_out = w.blk_de;
    VLA_TRY(gemm(r, "ex.time1", w.a, de, m->t1_w, H, de, de, et1, 0, frm(w.blk_de)));
    Epi et2 = epi_kind(EPI_F32, w.u, de, m->f32(m->t2_b));
    et2.blk_rows = blk;
    VLA_TRY(gemm(r, "ex.time2", w.hid, de, m->t2_w, H, de, de, et2, 0, frm(w.blk_de)));
    int pend = 0;
    for (int l = 0; l < c.ex_layers; ++l) {
      const void* K[MAX_ACT_BATCH] = {};
      const void* V[MAX_ACT_BATCH] = {};
      for (int f = 0; f < frames; ++f) {
        K[f] = (const char*)ctxs[f]->K + l * layer_k;
        V[f] = (const char*)ctxs[f]->V + l * layer_v;
      }
      VLA_TRY(decoder_layer(r, false, m->ex[l], w.u, H, de, c.ex_mlp, w.h, w.q, w.kown, w.vown, d.prefix,
                            K, V, d.prefix, w.att, w.mlp, false, &pend, frames, 0, 0,
                            fb ? &m->exw[l] : nullptr, l + 1 < c.ex_layers ? m->ex[l + 1].rms1 : m->fin_g));
    }
    // (pend < 0: the last down projection left h = x * fin_g and its row sums)
    if (pend >= 0) VLA_TRY(norm(r, w.u, frames * H, de, pend, nullptr, m->fin_g, -1, true, w.h, true, blk, w.blk_de));
    Epi e;
    if (pend < 0) fold_consumer(r, e, de);
    e.kind = EPI_EULER;
    e.afrag = 1;
    e.bias = m->f32(m->out_b);
    e.x = x;
    e.ldx = A;
    e.xop = w.xop;
    e.ldxop = d.a_pad;
    e.dt = m->step_b[k];
    e.xs = m->step_a[k];
    e.blk_rows = blk;
    e.blk_xop = w.blk_xop;
    VLA_TRY(gemm(r, "ex.out", w.h, de, m->out_w, H, A, de, e, 0, frm(w.blk_de)));
  }
  return VLA_OK;
}

static int run_denoise(const Run& r, const vla_ctx* ctx, const float* noise, float* x) {
  return run_denoise_n(r, &ctx, 1, noise, x);
}

// ---------------------------------------------------------------------------
// Creation
// ---------------------------------------------------------------------------

struct ScratchNeed {
  size_t floats = 0;
};

// (frames: up to that many frames' rows stacked, split-K planned for the
// rows plan_m (default: one frame's), for launches of up to plan_batch
// frames, as the launches plan them; the largest need over the frame counts)
static ScratchNeed gemm_scratch(int dt, int M, int N, int K, bool part = false, bool frag = false,
                                int frames = 1, int plan_batch = 1, int plan_m = 0) {
  ScratchNeed n{0};
  for (int f = 1; f <= frames; ++f) {
    GemmDesc g{dt, nullptr, K, nullptr, K, M * f, N, K, Epi()};
    g.plan_m = plan_m > 0 ? plan_m : M;
    g.plan_batch = plan_batch;
    if (part) g.epi.kind = EPI_PART;
    if (frag) g.frag_ks = (K + frag_slab(dt) - 1) / frag_slab(dt);
    n.floats = std::max(n.floats, plan_gemm(g).scratch_floats);
  }
  return n;
}

static ScratchNeed attn_scratch(int dt, int Sq, int nq, int nkv, int hd, int S0, int S1, int segs,
                                int plan_segs = 0) {
  AttnDesc a{};
  a.dtype = dt;
  a.Sq = Sq;
  a.nq = nq;
  a.nkv = nkv;
  a.hd = hd;
  a.S0 = S0;
  a.S1 = S1;
  a.segs = segs;
  a.plan_segs = plan_segs;
  return ScratchNeed{attn_scratch_floats(a)};
}

static int alloc_scratch(vla_model* m, const ScratchNeed& n, Scratch* s) {
  s->floats = std::max<size_t>(n.floats, 64);
  VLA_TRY(dmalloc(m, (void**)&s->ptr, s->floats * 4));
  return VLA_OK;
}

// RoPE tables [npos][hd / 2]: cos and sin of p 10000^(-2 i / hd), computed in
// fp64 and rounded to fp32.
static void rope_tables(int npos, int hd, std::vector<float>& cs, std::vector<float>& sn) {
  const int half = hd / 2;
  cs.assign((size_t)npos * half, 0.f);
  sn.assign((size_t)npos * half, 0.f);
  for (int p = 0; p < npos; ++p)
    for (int i = 0; i < half; ++i) {
      const double inv = std::pow(10000.0, -2.0 * i / hd);
      const double ang = p * inv;
      cs[(size_t)p * half + i] = (float)std::cos(ang);
      sn[(size_t)p * half + i] = (float)std::sin(ang);
    }
}

static int setup_tables(vla_model* m) {
  const vla_config& c = m->c;
  const Dims& d = m->d;
  const int npos = d.prefix + c.chunk_len;
  std::vector<float> cs, sn;
  rope_tables(npos, c.head_dim, cs, sn);
  VLA_TRY(dmalloc(m, (void**)&m->rope_cos, cs.size() * 4));
  VLA_TRY(dmalloc(m, (void**)&m->rope_sin, sn.size() * 4));
  HIP_TRY(hipMemcpy(m->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(m->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice));
  // sampler steps: Euler t_k = (N - k) / N in fp32, x += (-1/N) v; DDIM
  // (deterministic) over abar_s = prod_{i <= s} (1 - beta_i), beta linear on
  // [1e-4, 0.02] over 1000 training steps, timesteps s_k = floor((N - k)
  // 1000 / N) - 1, t_k = s_k / 1000, and x <- a_k x + b_k eps with
  // a_k = sqrt(abar_{k+1} / abar_k), b_k = sqrt(1 - abar_{k+1}) -
  // a_k sqrt(1 - abar_k) (abar after the last step = 1); coefficients in fp64
  m->step_a.assign(c.n_steps, 1.0f);
  m->step_b.assign(c.n_steps, -1.0f / (float)c.n_steps);
  m->step_t.resize(c.n_steps);
  if (c.sampler == VLA_SAMPLER_DDIM) {
    constexpr int TRAIN = 1000;
    std::vector<double> abar(TRAIN);
    double p = 1.0;
    for (int i = 0; i < TRAIN; ++i) {
      p *= 1.0 - (1e-4 + (0.02 - 1e-4) * i / (TRAIN - 1));
      abar[i] = p;
    }
    auto step_s = [&](int k) { return (c.n_steps - k) * TRAIN / c.n_steps - 1; };
    for (int k = 0; k < c.n_steps; ++k) {
      const double a0 = abar[step_s(k)], a1 = k + 1 < c.n_steps ? abar[step_s(k + 1)] : 1.0;
      const double a = std::sqrt(a1 / a0);
      m->step_a[k] = (float)a;
      m->step_b[k] = (float)(std::sqrt(1.0 - a1) - a * std::sqrt(1.0 - a0));
      m->step_t[k] = (float)step_s(k) / (float)TRAIN;
    }
  } else {
    for (int k = 0; k < c.n_steps; ++k) m->step_t[k] = (float)(c.n_steps - k) / (float)c.n_steps;
  }
  // sinusoid phi(t_k): periods log-spaced on [4e-3, 4]; the DiT's timestep
  // embedder takes a 256-wide phi
  const bool dit = c.head != VLA_HEAD_PI0;  // DiT and cognition-token heads: 256-wide phi, positions
  const int de = dit ? DIT_TIME_DIM : c.ex_dim, dh = de / 2;
  std::vector<float> phi((size_t)c.n_steps * de);
  for (int k = 0; k < c.n_steps; ++k) {
    const float t = m->step_t[k];
    for (int i = 0; i < dh; ++i) {
      const double frac = dh > 1 ? (double)i / (dh - 1) : 0.0;
      const double period = 4e-3 * std::pow(4.0 / 4e-3, frac);
      const double x = 2.0 * M_PI * (double)t / period;
      phi[(size_t)k * de + i] = (float)std::sin(x);
      phi[(size_t)k * de + dh + i] = (float)std::cos(x);
    }
  }
  // phi feeds a skinny GEMM: row-block operand layout (n_steps <= 64 rows)
  const size_t nphi = afrag_elems(m->dt, de);
  VLA_TRY(dmalloc(m, &m->phi, nphi * m->esz));
  if (m->dt == DT_BF16) {
    std::vector<uint16_t> hb(nphi, 0);
    for (int k = 0; k < c.n_steps; ++k)
      for (int i = 0; i < de; ++i) hb[afrag_index(m->dt, k, i)] = bf16_bits(phi[(size_t)k * de + i]);
    HIP_TRY(hipMemcpy(m->phi, hb.data(), hb.size() * 2, hipMemcpyHostToDevice));
  } else {
    std::vector<float> hf(nphi, 0.f);
    for (int k = 0; k < c.n_steps; ++k)
      for (int i = 0; i < de; ++i) hf[afrag_index(m->dt, k, i)] = phi[(size_t)k * de + i];
    HIP_TRY(hipMemcpy(m->phi, hf.data(), hf.size() * 4, hipMemcpyHostToDevice));
  }
  if (!dit) {
    VLA_TRY(dmalloc(m, (void**)&m->ck, (size_t)c.n_steps * de * 4));
    return VLA_OK;
  }
  // DiT: adaLN tables (filled at create) and the fixed token positions,
  // [sin(p w_i)]_i ++ [cos(p w_i)]_i with w_i = 10000^(-i / (d/2))
  const int dx = c.ex_dim, hx = dx / 2;
  if (c.head == VLA_HEAD_DIT) {
    VLA_TRY(dmalloc(m, (void**)&m->ada, (size_t)c.n_steps * c.ex_layers * 6 * dx * 4));
    VLA_TRY(dmalloc(m, (void**)&m->fada, (size_t)c.n_steps * 2 * dx * 4));
  } else {
    VLA_TRY(dmalloc(m, (void**)&m->ttok, (size_t)c.n_steps * dx * 4));
  }
  std::vector<float> pos((size_t)c.chunk_len * dx);
  for (int p = 0; p < c.chunk_len; ++p)
    for (int i = 0; i < hx; ++i) {
      const double ang = p * std::pow(10000.0, -(double)i / hx);
      pos[(size_t)p * dx + i] = (float)std::sin(ang);
      pos[(size_t)p * dx + hx + i] = (float)std::cos(ang);
    }
  VLA_TRY(dmalloc(m, (void**)&m->dpos, pos.size() * 4));
  HIP_TRY(hipMemcpy(m->dpos, pos.data(), pos.size() * 4, hipMemcpyHostToDevice));
  return VLA_OK;
}

// DiT: adaLN vectors of every step from the timestep embedder,
// W_l swish(W_t2 swish(W_t1 phi(t_k) + b_t1) + b_t2) + b_l (they depend on
// the step only), computed once with the library's GEMMs.
static int setup_dit_tables(vla_model* m) {
  const vla_config& c = m->c;
  const int de = c.ex_dim, N = c.n_steps, L = c.ex_layers;
  ActWs& w = *m->aws[0];
  Run r{m, nullptr, LaunchCaps{}, &w.scr, &w};
  Epi e1 = epi_kind(EPI_SWISH, w.a, de, m->f32(m->t1_b));
  e1.afrag = 1;
  VLA_TRY(gemm(r, "dit.time1", m->phi, DIT_TIME_DIM, m->t1_w, N, de, DIT_TIME_DIM, e1));
  Epi e2 = epi_kind(EPI_SWISH, w.hid, de, m->f32(m->t2_b));
  e2.afrag = 1;
  VLA_TRY(gemm(r, "dit.time2", w.a, de, m->t2_w, N, de, de, e2));
  for (int l = 0; l < L; ++l)
    VLA_TRY(gemm(r, "dit.ada", w.hid, de, m->dit[l].ada_w, N, 6 * de, de,
                 epi_kind(EPI_F32, m->ada + (size_t)l * 6 * de, L * 6 * de, m->f32(m->dit[l].ada_b))));
  VLA_TRY(gemm(r, "dit.ada", w.hid, de, m->fada_w, N, 2 * de, de,
               epi_kind(EPI_F32, m->fada, 2 * de, m->f32(m->fada_b))));
  return VLA_OK;
}

// Cognition-token head: the time token of every step, W_t2 swish(W_t1
// phi(t_k) + b_t1) + b_t2 (it depends on the step only), computed once with
// the library's GEMMs.
static int setup_cog_tables(vla_model* m) {
  const vla_config& c = m->c;
  const int de = c.ex_dim, N = c.n_steps;
  ActWs& w = *m->aws[0];
  Run r{m, nullptr, LaunchCaps{}, &w.scr, &w};
  Epi e1 = epi_kind(EPI_SWISH, w.a, de, m->f32(m->t1_b));
  e1.afrag = 1;
  VLA_TRY(gemm(r, "cog.time1", m->phi, DIT_TIME_DIM, m->t1_w, N, de, DIT_TIME_DIM, e1));
  VLA_TRY(gemm(r, "cog.time2", w.a, de, m->t2_w, N, de, de, epi_kind(EPI_F32, m->ttok, de, m->f32(m->t2_b))));
  return VLA_OK;
}

// One action lane's scratch (activations of the chunk rows, own K / V^T,
// partial sums, staging for graph replays).
static int add_act_lane(vla_model* m) {
  const vla_config& c = m->c;
  const Dims& d = m->d;
  const int dt = m->dt;
  const size_t e = m->esz;
  const int P = d.prefix, H = c.chunk_len, de = c.ex_dim, S = d.arows;
  auto upd = [](ScratchNeed& s, ScratchNeed x) { s.floats = std::max(s.floats, x.floats); };
  std::unique_ptr<ActWs> lane(new ActWs());
  ActWs& a = *lane;
  const int F = MAX_ACT_BATCH;
  const int qw = std::max(d.qd, de);  // query width (LM heads, or the DiT's)
  a.blk_xop = afrag_elems(dt, d.a_pad);
  a.blk_de = afrag_elems(dt, de);
  a.blk_att = afrag_elems(dt, qw);
  a.blk_mlp = afrag_elems(dt, c.ex_mlp);
  a.blk_k = own_k(m);
  a.blk_v = own_v(m);
  VLA_TRY(dmalloc(m, (void**)&a.u, (size_t)F * S * de * 4));
  // skinny-GEMM operands: row-block operand layout (64 rows per frame),
  // zeroed so the padding columns of xop stay zero
  VLA_TRY(dmalloc(m, &a.xop, F * a.blk_xop * e));
  HIP_TRY(hipMemset(a.xop, 0, F * a.blk_xop * e));
  VLA_TRY(dmalloc(m, &a.a, F * a.blk_de * e));
  VLA_TRY(dmalloc(m, &a.hid, F * a.blk_de * e));
  VLA_TRY(dmalloc(m, &a.h, F * a.blk_de * e));
  VLA_TRY(dmalloc(m, &a.q, (size_t)F * S * qw * e));
  VLA_TRY(dmalloc(m, &a.kown, F * a.blk_k * e));
  VLA_TRY(dmalloc(m, &a.vown, F * a.blk_v * e));
  HIP_TRY(hipMemset(a.kown, 0, F * a.blk_k * e));  // padding stays zero
  HIP_TRY(hipMemset(a.vown, 0, F * a.blk_v * e));
  VLA_TRY(dmalloc(m, &a.att, F * a.blk_att * e));
  VLA_TRY(dmalloc(m, &a.mlp, F * a.blk_mlp * e));
  ScratchNeed sa;
  if (c.head == VLA_HEAD_DIT) {
    const int N = c.n_steps;
    upd(sa, gemm_scratch(dt, H, de, d.a_pad, false, true));
    upd(sa, gemm_scratch(dt, N, de, DIT_TIME_DIM, false, true));
    upd(sa, gemm_scratch(dt, N, de, de, false, true));
    upd(sa, gemm_scratch(dt, N, 6 * de, de, false, true));
    upd(sa, gemm_scratch(dt, N, 2 * de, de, false, true));
    upd(sa, gemm_scratch(dt, H, de, de, false, true));
    upd(sa, gemm_scratch(dt, H, 3 * de, de, false, true));
    upd(sa, gemm_scratch(dt, H, de, de, true, true));
    upd(sa, gemm_scratch(dt, H, c.ex_mlp, de, false, true));
    upd(sa, gemm_scratch(dt, H, de, c.ex_mlp, true, true));
    upd(sa, gemm_scratch(dt, H, c.action_dim, de, false, true));
  }
  if (c.head == VLA_HEAD_COG) {
    const int N = c.n_steps;
    upd(sa, gemm_scratch(dt, H, de, d.a_pad, false, true));
    upd(sa, gemm_scratch(dt, N, de, DIT_TIME_DIM, false, true));
    upd(sa, gemm_scratch(dt, N, de, de, false, true));
    upd(sa, gemm_scratch(dt, S, 3 * de, de, false, true));
    upd(sa, gemm_scratch(dt, S, de, de, true, true));
    upd(sa, gemm_scratch(dt, S, c.ex_mlp, de, false, true));
    upd(sa, gemm_scratch(dt, S, de, c.ex_mlp, true, true));
    upd(sa, gemm_scratch(dt, H, c.action_dim, de, false, true));
  }
  // (split partials of all frames of a batched action phase)
  upd(sa, gemm_scratch(dt, F * H, de, d.a_pad, false, true));
  upd(sa, gemm_scratch(dt, F * H, de, de, false, true));
  upd(sa, gemm_scratch(dt, c.n_steps, de, de, false, true));
  upd(sa, gemm_scratch(dt, F * H, d.qkv_n, de, false, true));
  upd(sa, gemm_scratch(dt, F * H, de, d.qd, true, true));
  upd(sa, gemm_scratch(dt, F * H, 2 * c.ex_mlp, de, false, true));
  upd(sa, gemm_scratch(dt, F * H, de, c.ex_mlp, true, true));
  // batched loops: tiled GEMMs over all frames' rows, splits of one frame
  // (groups of 1 .. F frames, each planned for the largest group's rows)
  upd(sa, gemm_scratch(dt, H, d.qkv_n, de, false, false, F, 1, F * H));
  upd(sa, gemm_scratch(dt, H, de, d.qd, true, false, F, 1, F * H));
  upd(sa, gemm_scratch(dt, H, 2 * c.ex_mlp, de, false, false, F, 1, F * H));
  upd(sa, gemm_scratch(dt, H, de, c.ex_mlp, true, false, F, 1, F * H));
  upd(sa, gemm_scratch(dt, F * H, c.action_dim, de, false, true));
  upd(sa, attn_scratch(dt, H, c.lm_heads, c.lm_kv_heads, c.head_dim, P, H, 1));
  VLA_TRY(alloc_scratch(m, sa, &a.scr));
  {
    // the largest cache-attention launch of this head (all frames of a batched loop)
    int nc = 0;
    size_t nf = 0;
    if (c.head == VLA_HEAD_PI0)
      nf = attn_kv_split_floats(dt, F, H, c.lm_heads, c.lm_kv_heads, c.head_dim, P, H, &nc);
    else if (c.head == VLA_HEAD_DIT)
      nf = std::max(attn_kv_split_floats(dt, 1, H, c.ex_heads, c.ex_heads, d.ehd, P, 0, &nc),
                    attn_kv_split_floats(dt, 1, H, c.ex_heads, c.ex_heads, d.ehd, H, 0, &nc));
    else
      nf = attn_kv_split_floats(dt, 1, S, c.ex_heads, c.ex_heads, d.ehd, S, 0, &nc);
    if (c.head == VLA_HEAD_DIT) {  // counters for the larger of the two launches
      int n1 = 0, n2 = 0;
      attn_kv_split_floats(dt, 1, H, c.ex_heads, c.ex_heads, d.ehd, P, 0, &n1);
      attn_kv_split_floats(dt, 1, H, c.ex_heads, c.ex_heads, d.ehd, H, 0, &n2);
      nc = std::max(n1, n2);
    }
    if (nf) {
      VLA_TRY(dmalloc(m, (void**)&a.apart, nf * 4));
      a.apart_floats = nf;
      VLA_TRY(dmalloc(m, (void**)&a.acnt, (size_t)std::max(nc, 1) * 4));
      HIP_TRY(hipMemset(a.acnt, 0, (size_t)std::max(nc, 1) * 4));
      a.acnt_n = nc;
    }
  }
  if (c.head == VLA_HEAD_PI0 && (c.ex_dim + 31) / 32 <= FOLD_MAX_PAIRS && c.ex_dim % 8 == 0 && H <= 64) {
    VLA_TRY(dmalloc(m, (void**)&a.rowss, (size_t)FOLD_MAX_PAIRS * 64 * 4));
    VLA_TRY(dmalloc(m, (void**)&a.pcnt, (size_t)FOLD_MAX_PAIRS * 4));
    HIP_TRY(hipMemset(a.pcnt, 0, (size_t)FOLD_MAX_PAIRS * 4));
  }
  VLA_TRY(dmalloc(m, (void**)&a.xg, (size_t)F * H * c.action_dim * 4));
  VLA_TRY(dmalloc(m, (void**)&a.nstage, (size_t)F * H * c.action_dim * 4));
  m->aws.push_back(std::move(lane));
  return VLA_OK;
}

// A VLM lane for up to `cap` frames per prefill. Lane `slot` is replaced when
// it exists (after the device is idle); its cached prefill graphs go with it.
static int make_vlm_lane(vla_model* m, int cap, int slot) {
  const vla_config& c = m->c;
  const Dims& d = m->d;
  const int dt = m->dt;
  const size_t e = m->esz;
  const size_t rv = (size_t)cap * d.rows_v, P = (size_t)cap * d.prefix;
  const int dv = c.vit_dim, dl = c.lm_dim;
  std::unique_ptr<VlmWs> lane(new VlmWs());
  VlmWs& v = *lane;
  v.cap = cap;
  auto alloc = [&](void** p, size_t bytes) {
    hipError_t err = hipMalloc(p, std::max<size_t>(bytes, 256));
    if (err != hipSuccess) return fail(VLA_ENOMEM, std::string("hipMalloc: ") + hipGetErrorString(err));
    v.mem.push_back(*p);
    return VLA_OK;
  };
  const size_t rmax = std::max(rv, P);
  VLA_TRY(alloc((void**)&v.xv, rv * dv * 4));
  VLA_TRY(alloc((void**)&v.xl, P * dl * 4));
  VLA_TRY(alloc(&v.h, rmax * std::max({d.kp_pad, dv, dl}) * e));
  VLA_TRY(alloc(&v.qkv, std::max(rv * 3 * dv, P * d.qd) * e));
  VLA_TRY(alloc(&v.att, std::max(rv * dv, P * d.qd) * e));
  VLA_TRY(alloc(&v.mlp, std::max(rv * c.vit_mlp, P * c.lm_mlp) * e));
  VLA_TRY(alloc(&v.sbuf, (size_t)cap * d.s_pad * e));
  // split partials of all frames' rows (splits planned for one frame)
  ScratchNeed sv;
  auto upd = [](ScratchNeed& s, ScratchNeed x) { s.floats = std::max(s.floats, x.floats); };
  const int r1 = d.rows_v, p1 = d.prefix;
  upd(sv, gemm_scratch(dt, r1, dv, d.kp_pad, false, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, r1, 3 * dv, dv, false, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, r1, dv, dv, true, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, r1, c.vit_mlp, dv, false, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, r1, dv, c.vit_mlp, true, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, d.nimg, dl, d.kproj));
  if (c.head == VLA_HEAD_DIT) upd(sv, gemm_scratch(dt, p1, 2 * c.ex_dim, dl, false, false, cap, MAX_VLM_BATCH));
  if (c.head == VLA_HEAD_COG) upd(sv, gemm_scratch(dt, 1, c.ex_dim, dl));
  upd(sv, gemm_scratch(dt, 1, dl, d.s_pad));
  upd(sv, gemm_scratch(dt, p1, d.qkv_n, dl, false, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, p1, dl, d.qd, true, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, p1, 2 * c.lm_mlp, dl, false, false, cap, MAX_VLM_BATCH));
  upd(sv, gemm_scratch(dt, p1, dl, c.lm_mlp, true, false, cap, MAX_VLM_BATCH));
  upd(sv, attn_scratch(dt, d.tview, c.vit_heads, c.vit_heads, d.vhd, d.tview, 0, cap * c.n_views, c.n_views));
  upd(sv, attn_scratch(dt, p1, c.lm_heads, c.lm_kv_heads, c.head_dim, p1, 0, 1));
  if (sv.floats) {
    VLA_TRY(alloc((void**)&v.scr.ptr, sv.floats * 4));
    v.scr.floats = sv.floats;
  }
  VLA_TRY(alloc((void**)&v.pstage, (size_t)cap * c.n_views * c.img_h * c.img_w * 3 * 4));
  VLA_TRY(alloc((void**)&v.istage, (size_t)cap * std::max(c.n_text, 1) * 4));
  VLA_TRY(alloc((void**)&v.sstage, (size_t)cap * std::max(c.state_dim, 1) * 4));
  if (slot < (int)m->vws.size()) {
    HIP_TRY(hipDeviceSynchronize());
    for (auto it = m->pre_graphs.begin(); it != m->pre_graphs.end();) {
      if (std::get<0>(it->first) == slot) {
        hipGraphExecDestroy(it->second);
        it = m->pre_graphs.erase(it);
      } else {
        ++it;
      }
    }
    m->vws[slot] = std::move(lane);
  } else {
    m->vws.push_back(std::move(lane));
  }
  return VLA_OK;
}

static int add_vlm_lane(vla_model* m) { return make_vlm_lane(m, 1, (int)m->vws.size()); }

static int setup_workspaces(vla_model* m) {
  VLA_TRY(add_vlm_lane(m));
  VLA_TRY(add_act_lane(m));
  return VLA_OK;
}

static int create_impl(const vla_config* cfg, uint64_t seed, vla_model** out) {
  VLA_TRY(validate(cfg));
  std::unique_ptr<vla_model> m(new vla_model());
  m->c = *cfg;
  m->d = derive(*cfg);
  m->dt = cfg->dtype == VLA_BF16 ? DT_BF16 : DT_F32;
  m->esz = dsz(m->dt);
  m->seed = seed;
  HIP_TRY(hipGetDevice(&m->device));
  hipDeviceProp_t prop;
  HIP_TRY(hipGetDeviceProperties(&prop, m->device));
  m->num_cus = prop.multiProcessorCount;
  build_inventory(m.get());
  size_t off = 0;
  for (auto& t : m->T) {
    t.offset = off;
    off += (t.bytes() + 255) / 256 * 256;
  }
  m->arena_bytes = off;
  hipError_t e = hipMalloc(&m->arena, off);
  if (e != hipSuccess) return fail(VLA_ENOMEM, std::string("weights: hipMalloc: ") + hipGetErrorString(e));
  std::vector<std::vector<int>> by_tensor(m->T.size());
  for (size_t i = 0; i < m->P.size(); ++i) by_tensor[m->P[i].tensor].push_back((int)i);
  for (size_t t = 0; t < m->T.size(); ++t) {
    int rc = upload_tensor(m.get(), (int)t, by_tensor[t]);
    if (rc != VLA_OK) {
      hipFree(m->arena);
      return rc;
    }
  }
  int rc = setup_tables(m.get());
  if (rc == VLA_OK) rc = setup_workspaces(m.get());
  if (rc == VLA_OK && m->c.head == VLA_HEAD_DIT) {
    rc = setup_dit_tables(m.get());
  } else if (rc == VLA_OK && m->c.head == VLA_HEAD_COG) {
    rc = setup_cog_tables(m.get());
  } else if (rc == VLA_OK) {
    // c_k = W_2[:, d_e:] phi(t_k) + b_2 for every step (depends on the step only)
    Run r{m.get(), nullptr, LaunchCaps{}, &m->aws[0]->scr, m->aws[0].get()};
    const int de = m->c.ex_dim;
    rc = gemm(r, "ex.ck", m->phi, de, m->t1_w, m->c.n_steps, de, de,
              epi_kind(EPI_F32, m->ck, de, m->f32(m->t1_b)), de);
  }
  if (rc == VLA_OK) {
    hipError_t se = hipDeviceSynchronize();
    if (se != hipSuccess) rc = fail(VLA_EHIP, std::string("create: ") + hipGetErrorString(se));
  }
  if (rc != VLA_OK) {
    for (void* p : m->allocs) hipFree(p);
    hipFree(m->exw_mem);
    hipFree(m->arena);
    return rc;
  }
  *out = m.release();
  return VLA_OK;
}

// ---------------------------------------------------------------------------
// Pipeline
// ---------------------------------------------------------------------------

static void ctx_free(vla_ctx* c) {
  if (!c) return;
  if (c->own) {
    hipFree(c->K);
    hipFree(c->V);
    hipFree(c->XK);
    hipFree(c->XV);
    hipFree(c->cog);
  }
  delete c;
}

// n contexts whose buffers are consecutive slices of one zeroed allocation
// each (context i at i times the context size), so a batched prefill reaches
// frame i's cache at a fixed stride. out[0] owns the allocations.
static int ctx_create_n(vla_model* m, int n, vla_ctx** out) {
  const size_t kb = ctx_kbytes(m), vb = ctx_vbytes(m), xb = ctx_xbytes(m);
  const size_t cb = m->c.head == VLA_HEAD_COG ? (size_t)m->c.ex_dim * 4 : 0;
  void *K = nullptr, *V = nullptr, *XK = nullptr, *XV = nullptr, *CG = nullptr;
  auto zalloc = [](void** p, size_t bytes) {
    hipError_t e = hipMalloc(p, bytes);
    if (e == hipSuccess) e = hipMemset(*p, 0, bytes);  // padding stays zero
    return e;
  };
  hipError_t e = zalloc(&K, n * kb);
  if (e == hipSuccess) e = zalloc(&V, n * vb);
  if (e == hipSuccess && xb) e = zalloc(&XK, n * xb);
  if (e == hipSuccess && xb) e = zalloc(&XV, n * xb);
  if (e == hipSuccess && cb) e = zalloc(&CG, n * cb);
  if (e != hipSuccess) {
    hipFree(K);
    hipFree(V);
    hipFree(XK);
    hipFree(XV);
    hipFree(CG);
    return fail(VLA_ENOMEM, std::string("context buffers: ") + hipGetErrorString(e));
  }
  for (int i = 0; i < n; ++i) {
    vla_ctx* c = new vla_ctx();
    c->m = m;
    c->own = i == 0;
    c->K = (char*)K + i * kb;
    c->V = (char*)V + i * vb;
    c->XK = xb ? (char*)XK + i * xb : nullptr;
    c->XV = xb ? (char*)XV + i * xb : nullptr;
    c->cog = cb ? (float*)((char*)CG + i * cb) : nullptr;
    out[i] = c;
  }
  return VLA_OK;
}

static int ctx_create_impl(vla_model* m, vla_ctx** out) { return ctx_create_n(m, 1, out); }

static void cu_mask(int first, int count, int total, std::vector<uint32_t>& mask) {
  mask.assign((total + 31) / 32, 0u);
  for (int i = first; i < first + count && i < total; ++i) mask[i / 32] |= 1u << (i % 32);
}

static int get_streams(vla_model* m, const vla_sched& s, Streams* out) {
  if (s.mode == VLA_MODE_CU_MASKED) {
    auto key = std::make_pair(s.vlm_cus, s.act_cus);
    auto it = m->mask_streams.find(key);
    if (it == m->mask_streams.end()) {
      // Bits are spread over the XCDs by the driver (bit i -> XCD i % 8), so
      // contiguous ranges whose sizes are multiples of 8 give every XCD CUs
      // of both phases. All action streams share the action CU set.
      Streams st;
      std::vector<uint32_t> mv, ma;
      cu_mask(0, s.vlm_cus, m->num_cus, mv);
      cu_mask(s.vlm_cus, s.act_cus, m->num_cus, ma);
      // creation order: as for the plain streams below
      HIP_TRY(hipExtStreamCreateWithCUMask(&st.v[0], (uint32_t)mv.size(), mv.data()));
      for (int i = 0; i < 2; ++i)
        HIP_TRY(hipExtStreamCreateWithCUMask(&st.a[i], (uint32_t)ma.size(), ma.data()));
      for (int i = 2; i < MAX_ACT_STREAMS; ++i)
        HIP_TRY(hipExtStreamCreateWithCUMask(&st.a[i], (uint32_t)ma.size(), ma.data()));
      for (int i = 1; i < MAX_VLM_STREAMS; ++i)
        HIP_TRY(hipExtStreamCreateWithCUMask(&st.v[i], (uint32_t)mv.size(), mv.data()));
      it = m->mask_streams.emplace(key, st).first;
    }
    *out = it->second;
    return VLA_OK;
  }
  if (!m->plain.v[0]) {
    // The HIP runtime maps streams onto a few hardware queues (4 per process
    // unless GPU_MAX_HW_QUEUES says otherwise) and later streams share them.
    // The first VLM stream and the first two action streams are created
    // first, so the common schedules (one VLM lane, one or two action lanes)
    // get hardware queues of their own next to the default stream's.
    HIP_TRY(hipStreamCreateWithFlags(&m->plain.v[0], hipStreamNonBlocking));
    for (int i = 0; i < 2; ++i) HIP_TRY(hipStreamCreateWithFlags(&m->plain.a[i], hipStreamNonBlocking));
    for (int i = 2; i < MAX_ACT_STREAMS; ++i)
      HIP_TRY(hipStreamCreateWithFlags(&m->plain.a[i], hipStreamNonBlocking));
    for (int i = 1; i < MAX_VLM_STREAMS; ++i)
      HIP_TRY(hipStreamCreateWithFlags(&m->plain.v[i], hipStreamNonBlocking));
  }
  *out = m->plain;
  return VLA_OK;
}

// Capture one phase on `st` into an executable graph.
template <typename F>
static int capture(hipStream_t st, F&& body, hipGraphExec_t* out) {
  HIP_TRY(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
  const int rc = body();
  hipGraph_t g = nullptr;
  const hipError_t e = hipStreamEndCapture(st, &g);
  if (rc != VLA_OK) {
    if (g) hipGraphDestroy(g);
    return rc;
  }
  if (e != hipSuccess) return fail(VLA_EHIP, std::string("graph capture: ") + hipGetErrorString(e));
  const hipError_t ie = hipGraphInstantiate(out, g, nullptr, nullptr, 0);
  hipGraphDestroy(g);
  if (ie != hipSuccess) return fail(VLA_EHIP, std::string("graph instantiate: ") + hipGetErrorString(ie));
  return VLA_OK;
}

static int pipeline_impl(vla_model* m, const vla_frame* frames, const float* noise, int R,
                         const vla_sched* sched, float* actions, vla_timing* t) {
  if (!frames || !noise || !actions || !sched) return fail(VLA_EINVAL, "NULL argument");
  if (R < 1) return fail(VLA_EINVAL, "R must be >= 1");
  const vla_sched& s = *sched;
  if (s.mode < VLA_MODE_SERIAL || s.mode > VLA_MODE_WG_CAPPED) return fail(VLA_EINVAL, "unknown mode");
  if (s.mode == VLA_MODE_CU_MASKED) {
    if (s.vlm_cus <= 0 || s.act_cus <= 0 || s.vlm_cus % 8 || s.act_cus % 8 ||
        s.vlm_cus + s.act_cus > m->num_cus)
      return fail(VLA_EINVAL, "CU split: both counts positive multiples of 8, sum <= CU count (" +
                                  std::to_string(m->num_cus) + ")");
  }
  if (s.mode == VLA_MODE_WG_CAPPED && s.vlm_wg_cap < 1) return fail(VLA_EINVAL, "vlm_wg_cap must be >= 1");
  const int lanes = std::max(1, s.act_streams);
  if (lanes > MAX_ACT_STREAMS) return fail(VLA_EINVAL, "act_streams must be <= 4");
  if (lanes > 1 && s.mode == VLA_MODE_SERIAL) return fail(VLA_EINVAL, "act_streams > 1 needs a concurrent mode");
  const int vlanes = std::max(1, s.vlm_streams);
  if (vlanes > MAX_VLM_STREAMS) return fail(VLA_EINVAL, "vlm_streams must be <= 2");
  if (vlanes > 1 && s.mode == VLA_MODE_SERIAL) return fail(VLA_EINVAL, "vlm_streams > 1 needs a concurrent mode");
  const int B = std::max(1, s.act_batch);
  if (B > MAX_ACT_BATCH) return fail(VLA_EINVAL, "act_batch must be <= " + std::to_string(MAX_ACT_BATCH));
  if (B > 1 && m->c.head != VLA_HEAD_PI0) return fail(VLA_EINVAL, "act_batch > 1: pi0-style action head only");
  if (s.act_chunks < 0 || s.act_chunks > 64) return fail(VLA_EINVAL, "act_chunks must be in 0 .. 64");
  const int Bv = std::max(1, s.vlm_batch);
  if (Bv > MAX_VLM_BATCH || CTX_BLOCK % Bv) return fail(VLA_EINVAL, "vlm_batch must be 1, 2, 4 or 8");
  const vla_config& c = m->c;
  for (int r = 0; r < R; ++r)
    if (!frames[r].pixels || (c.n_text > 0 && !frames[r].text_ids) || (c.state_dim > 0 && !frames[r].state))
      return fail(VLA_EINVAL, "frame " + std::to_string(r) + " has a NULL input");
  std::lock_guard<std::mutex> lock(m->mu);
  // A context is in flight from its prefill until its action phase ends.
  // Prefills go in groups of Bv consecutive frames (consecutive contexts of
  // one block), action phases in groups of B. The ring holds whole blocks and
  // at least Bv + B contexts, so a prefill only ever waits for action phases
  // of frames before its own group.
  const int nctx = rnd_up(Bv * vlanes + B * lanes + std::max(Bv, B), CTX_BLOCK);
  while ((int)m->pctx.size() < nctx) {
    vla_ctx* blk[CTX_BLOCK];
    VLA_TRY(ctx_create_n(m, CTX_BLOCK, blk));
    for (vla_ctx* cx : blk) m->pctx.push_back(cx);
  }
  while ((int)m->aws.size() < lanes) VLA_TRY(add_act_lane(m));
  for (int vi = 0; vi < vlanes; ++vi)
    if (vi >= (int)m->vws.size() || m->vws[vi]->cap < Bv) VLA_TRY(make_vlm_lane(m, Bv, vi));
  if (B > 1) VLA_TRY(ensure_wide(m));
  Streams st;
  VLA_TRY(get_streams(m, s, &st));
  if (s.mode == VLA_MODE_SERIAL) st.a[0] = st.v[0];
  const bool graphs = s.graphs != 0 && m->timer_tag.empty();
  // Asynchronous inference: k action chunks (items) per VLM output. Item i
  // is chunk i % k of frame i / k, with its own noise and output rows.
  const int k = std::max(1, s.act_chunks);
  const int items = R * k;
  auto grow = [&](std::vector<hipEvent_t>& v, size_t n) -> int {
    while (v.size() < n) {
      hipEvent_t e;
      HIP_TRY(hipEventCreate(&e));
      v.push_back(e);
    }
    return VLA_OK;
  };
  // events: ev[2r] / ev[2r+1] VLM start / end of frame r; eva[2i] / eva[2i+1]
  // action start / end of item i. A group's time is recorded on its first
  // member, the others get an empty interval at the group's end; a frame's
  // context is free again at the end event of its last item.
  VLA_TRY(grow(m->ev, (size_t)2 * R));
  VLA_TRY(grow(m->eva, (size_t)2 * items));
  LaunchCaps vcaps{}, acaps{};
  if (s.mode == VLA_MODE_WG_CAPPED) vcaps.max_wgs = s.vlm_wg_cap * m->num_cus;
  const size_t chunk = (size_t)c.chunk_len * c.action_dim;
  const size_t pix_bytes = (size_t)c.n_views * c.img_h * c.img_w * 3 * 4;
  auto vlane = [&](int r) { return (r / Bv) % vlanes; };  // VLM lane of frame r
  auto alane = [&](int i) { return (i / B) % lanes; };    // action lane of item i
  auto actx = [&](int i) { return (i / k) % nctx; };      // context of item i
  HIP_TRY(hipDeviceSynchronize());

  auto den_key = [&](int li, int a0, int na) {
    std::vector<int> cs;
    for (int f = 0; f < na; ++f) cs.push_back(actx(a0 + f));
    return std::make_pair(li, cs);
  };
  if (graphs) {  // capture what this run needs and is missing (outside the timed loop)
    for (int g0 = 0; g0 < R; g0 += Bv) {
      const int n = std::min(Bv, R - g0), vi = vlane(g0), ci = g0 % nctx;
      const auto key = std::make_tuple(vi, ci, vcaps.max_wgs, n);
      if (m->pre_graphs.count(key)) continue;
      VlmWs* vw = m->vws[vi].get();
      vla_frame staged[MAX_VLM_BATCH];
      for (int i = 0; i < n; ++i)
        staged[i] = vla_frame{vw->pstage + i * pix_bytes / 4, vw->istage + (size_t)i * std::max(c.n_text, 1),
                              c.state_dim > 0 ? vw->sstage + (size_t)i * c.state_dim : nullptr};
      Run rv{m, st.v[vi], vcaps, &vw->scr, nullptr, vw};
      hipGraphExec_t ge = nullptr;
      VLA_TRY(capture(st.v[vi], [&] { return run_prefill_n(rv, staged, n, &m->pctx[ci]); }, &ge));
      m->pre_graphs[key] = ge;
    }
    // one graph per (lane, contexts of the group's items)
    for (int a0 = 0; a0 < items; a0 += B) {
      const int na = std::min(B, items - a0), li = alane(a0);
      const auto key = den_key(li, a0, na);
      if (m->den_graphs.count(key)) continue;
      ActWs* aw = m->aws[li].get();
      Run ra{m, st.a[li], acaps, &aw->scr, aw};
      const vla_ctx* cs[MAX_ACT_BATCH] = {};
      for (int f = 0; f < na; ++f) cs[f] = m->pctx[actx(a0 + f)];
      hipGraphExec_t ge = nullptr;
      VLA_TRY(capture(st.a[li], [&] { return run_denoise_n(ra, cs, na, aw->nstage, aw->xg); }, &ge));
      m->den_graphs[key] = ge;
    }
  }

  const auto t0 = std::chrono::steady_clock::now();
  int next_item = 0;  // first item whose action phase is not issued yet
  for (int g0 = 0; g0 < R; g0 += Bv) {
    const int n = std::min(Bv, R - g0), vi = vlane(g0), ci = g0 % nctx;
    hipStream_t sv = st.v[vi];
    VlmWs* vw = m->vws[vi].get();
    // a context is free once the action phases that read it are done
    for (int q = g0; q < g0 + n; ++q) {
      if (q < nctx) continue;
      const int last = (q - nctx) * k + k - 1;  // the previous user's last item
      if (sv != st.a[alane(last)]) HIP_TRY(hipStreamWaitEvent(sv, m->eva[2 * last + 1], 0));
    }
    HIP_TRY(hipEventRecord(m->ev[2 * g0], sv));
    if (graphs) {
      for (int i = 0; i < n; ++i) {
        const vla_frame& fr = frames[g0 + i];
        HIP_TRY(launch_copy(vw->pstage + i * pix_bytes / 4, fr.pixels, pix_bytes, sv));
        if (c.n_text > 0)
          HIP_TRY(launch_copy(vw->istage + (size_t)i * c.n_text, fr.text_ids, (size_t)c.n_text * 4, sv));
        if (c.state_dim > 0)
          HIP_TRY(launch_copy(vw->sstage + (size_t)i * c.state_dim, fr.state, (size_t)c.state_dim * 4, sv));
      }
      HIP_TRY(hipGraphLaunch(m->pre_graphs[std::make_tuple(vi, ci, vcaps.max_wgs, n)], sv));
    } else {
      Run rv{m, sv, vcaps, &vw->scr, nullptr, vw};
      VLA_TRY(run_prefill_n(rv, &frames[g0], n, &m->pctx[ci]));
    }
    HIP_TRY(hipEventRecord(m->ev[2 * g0 + 1], sv));
    for (int q = g0 + 1; q < g0 + n; ++q) {
      HIP_TRY(hipEventRecord(m->ev[2 * q], sv));
      HIP_TRY(hipEventRecord(m->ev[2 * q + 1], sv));
    }
    // every action group whose frames are all prefilled starts now
    while (next_item < items) {
      const int a0 = next_item, na = std::min(B, items - a0);
      const int f_first = a0 / k, f_last = (a0 + na - 1) / k;
      if (f_last >= g0 + n) break;
      next_item += na;
      const int li = alane(a0);
      hipStream_t sa = st.a[li];
      for (int q = f_first; q <= f_last; ++q)
        if (st.v[vlane(q)] != sa) HIP_TRY(hipStreamWaitEvent(sa, m->ev[2 * q + 1], 0));
      HIP_TRY(hipEventRecord(m->eva[2 * a0], sa));
      ActWs* aw = m->aws[li].get();
      if (graphs) {
        HIP_TRY(launch_copy(aw->nstage, noise + a0 * chunk, na * chunk * 4, sa));
        HIP_TRY(hipGraphLaunch(m->den_graphs[den_key(li, a0, na)], sa));
        HIP_TRY(launch_copy(actions + a0 * chunk, aw->xg, na * chunk * 4, sa));
      } else {
        Run ra{m, sa, acaps, &aw->scr, aw};
        const vla_ctx* cs[MAX_ACT_BATCH] = {};
        for (int f = 0; f < na; ++f) cs[f] = m->pctx[actx(a0 + f)];
        VLA_TRY(run_denoise_n(ra, cs, na, noise + a0 * chunk, actions + a0 * chunk));
      }
      HIP_TRY(hipEventRecord(m->eva[2 * a0 + 1], sa));
      for (int q = a0 + 1; q < a0 + na; ++q) {
        HIP_TRY(hipEventRecord(m->eva[2 * q], sa));
        HIP_TRY(hipEventRecord(m->eva[2 * q + 1], sa));
      }
    }
  }
  for (int vi = 0; vi < vlanes; ++vi) HIP_TRY(hipStreamSynchronize(st.v[vi]));
  for (int li = 0; li < lanes; ++li) HIP_TRY(hipStreamSynchronize(st.a[li]));
  const auto t1 = std::chrono::steady_clock::now();
  if (t) {
    t->wall_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
    t->frames_per_s = R / (t->wall_ms * 1e-3);
    t->actions_per_s = t->frames_per_s * k * c.chunk_len;
    t->vlm_ms = t->act_ms = 0;
    for (int r = 0; r < R; ++r) {
      float a = 0;
      HIP_TRY(hipEventElapsedTime(&a, m->ev[2 * r], m->ev[2 * r + 1]));
      t->vlm_ms += a;
    }
    for (int i = 0; i < items; ++i) {
      float b = 0;
      HIP_TRY(hipEventElapsedTime(&b, m->eva[2 * i], m->eva[2 * i + 1]));
      t->act_ms += b;
    }
  }
  return VLA_OK;
}

// ---------------------------------------------------------------------------
// Allocation-free GEMM: split-K partials in a fixed device array
// ---------------------------------------------------------------------------

// Split-K partials of vla_gemm_noalloc. Every GPU the library runs on holds
// its own copy until the process ends. In host code `scratch` only names the
// symbol: kernels get the device address that hipGetSymbolAddress returns
// for the current device (noalloc_scratch below), never the name itself.
constexpr size_t NOALLOC_SCRATCH_FLOATS = (size_t)2 << 20;  // 8 MiB
static __device__ __align__(256) float scratch[NOALLOC_SCRATCH_FLOATS];

constexpr int NOALLOC_MAX_DEVICES = 64;
static float* g_noalloc_ptr[NOALLOC_MAX_DEVICES] = {};
static std::mutex g_noalloc_mu;

// Device address of the current device's copy of `scratch`, looked up on the
// first call on that device (with it current) and kept.
static int noalloc_scratch(float** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return fail(VLA_EUNSUPPORTED, "device index above 63");
  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  if (!g_noalloc_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(VLA_EHIP, "hipGetSymbolAddress returned NULL for the scratch array");
    g_noalloc_ptr[dev] = (float*)p;
  }
  *out = g_noalloc_ptr[dev];
  return VLA_OK;
}

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------

// No C++ exception crosses the ABI: an allocation failure is VLA_ENOMEM,
// any other exception (a library defect, not a caller error) VLA_ESTATE.
#define ABI_GUARD(...)                                                          \
  try {                                                                         \
    g_err.clear();                                                              \
    __VA_ARGS__                                                                 \
  } catch (const std::bad_alloc& ex) {                                          \
    return fail(VLA_ENOMEM, std::string("host allocation failed: ") + ex.what()); \
  } catch (const std::exception& ex) {                                          \
    return fail(VLA_ESTATE, std::string("internal exception: ") + ex.what());   \
  } catch (...) {                                                               \
    return fail(VLA_ESTATE, "internal exception");                              \
  }

extern "C" {

const char* vla_last_error(void) { return g_err.c_str(); }

int vla_preset(const char* name, vla_config* out) {
  ABI_GUARD({
    if (!preset(name, out)) return fail(VLA_EINVAL, std::string("unknown preset ") + (name ? name : "(null)"));
    return VLA_OK;
  })
}

int vla_validate(const vla_config* cfg) { ABI_GUARD({ return validate(cfg); }) }

int vla_create(const vla_config* cfg, uint64_t seed, vla_model** out) {
  ABI_GUARD({
    if (!out) return fail(VLA_EINVAL, "out is NULL");
    *out = nullptr;
    return create_impl(cfg, seed, out);
  })
}

int vla_model_config(const vla_model* m, vla_config* out) {
  ABI_GUARD({
    if (!m || !out) return fail(VLA_EINVAL, "NULL argument");
    *out = m->c;
    return VLA_OK;
  })
}

int vla_destroy(vla_model* m) {
  ABI_GUARD({
    if (!m) return VLA_OK;
    hipDeviceSynchronize();
    for (auto& kv : m->pre_graphs) hipGraphExecDestroy(kv.second);
    for (auto& kv : m->den_graphs) hipGraphExecDestroy(kv.second);
    // members of a block first, its owner last
    for (auto it = m->pctx.rbegin(); it != m->pctx.rend(); ++it) ctx_free(*it);
    auto drop = [](Streams& st) {
      for (hipStream_t v : st.v)
        if (v) hipStreamDestroy(v);
      for (hipStream_t a : st.a)
        if (a) hipStreamDestroy(a);
    };
    for (auto& kv : m->mask_streams) drop(kv.second);
    drop(m->plain);
    for (auto e : m->ev) hipEventDestroy(e);
    for (auto e : m->eva) hipEventDestroy(e);
    for (auto e : m->timer_ev) hipEventDestroy(e);
    for (auto& so : m->solo)
      if (so.done) hipEventDestroy(so.done);
    if (m->wlog) {
      wavelog_set(nullptr);
      hipFree(m->wlog);
    }
    for (void* p : m->allocs) hipFree(p);
    hipFree(m->exw_mem);
    hipFree(m->arena);
    delete m;
    return VLA_OK;
  })
}

int vla_ctx_create(vla_model* m, vla_ctx** out) {
  ABI_GUARD({
    if (!m || !out) return fail(VLA_EINVAL, "NULL argument");
    *out = nullptr;
    return ctx_create_impl(m, out);
  })
}

int vla_ctx_destroy(vla_ctx* c) {
  ABI_GUARD({
    if (!c) return VLA_OK;
    ctx_free(c);
    return VLA_OK;
  })
}

// Orders standalone calls of one phase: a call on another stream than the
// previous one waits (on the device) for that call's work, so the two never
// share the lane-0 scratch at once. Under stream capture the call is neither
// ordered nor recorded (an event recorded outside the capture cannot be
// waited on inside it); captured calls on several streams still race.
static hipError_t solo_begin(vla_model* m, int phase, hipStream_t st, bool* capturing) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(st, &cs);
  if (e != hipSuccess) return e;
  *capturing = cs != hipStreamCaptureStatusNone;
  auto& s = m->solo[phase];
  if (*capturing) {
    s.pending = false;
    return hipSuccess;
  }
  if (!s.done && (e = hipEventCreateWithFlags(&s.done, hipEventDisableTiming)) != hipSuccess) return e;
  if (s.pending && s.stream != st && (e = hipStreamWaitEvent(st, s.done, 0)) != hipSuccess) return e;
  return hipSuccess;
}

static hipError_t solo_end(vla_model* m, int phase, hipStream_t st, bool capturing) {
  auto& s = m->solo[phase];
  if (capturing) return hipSuccess;
  const hipError_t e = hipEventRecord(s.done, st);
  s.stream = st;
  s.pending = e == hipSuccess;
  return e;
}

// host wait for the last standalone call of each phase (the pipeline reuses
// the lane-0 scratch)
static hipError_t solo_drain(vla_model* m) {
  for (auto& s : m->solo)
    if (s.pending) {
      const hipError_t e = hipEventSynchronize(s.done);
      if (e != hipSuccess) return e;
      s.pending = false;
    }
  return hipSuccess;
}

int vla_vlm_prefill(vla_model* m, const vla_frame* in, vla_ctx* ctx, void* stream) {
  ABI_GUARD({
    if (!m || !in || !ctx || !in->pixels || (!in->text_ids && m->c.n_text > 0))
      return fail(VLA_EINVAL, "NULL argument");
    if (m->c.state_dim > 0 && !in->state) return fail(VLA_EINVAL, "state is NULL but state_dim > 0");
    if (ctx->m != m) return fail(VLA_ESTATE, "context belongs to another model");
    bool cap = false;
    hipError_t e = solo_begin(m, 0, (hipStream_t)stream, &cap);
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("ordering standalone prefills: ") + hipGetErrorString(e));
    Run r{m, (hipStream_t)stream, LaunchCaps{}, &m->vws[0]->scr, nullptr, m->vws[0].get()};
    const int rc = run_prefill(r, in, ctx);
    e = solo_end(m, 0, (hipStream_t)stream, cap);
    if (rc == VLA_OK && e != hipSuccess) return fail(VLA_EHIP, std::string("ordering standalone prefills: ") + hipGetErrorString(e));
    return rc;
  })
}

int vla_action_denoise(vla_model* m, const vla_ctx* ctx, const float* noise, float* actions, void* stream) {
  ABI_GUARD({
    if (!m || !ctx || !noise || !actions) return fail(VLA_EINVAL, "NULL argument");
    if (ctx->m != m) return fail(VLA_ESTATE, "context belongs to another model");
    bool cap = false;
    hipError_t e = solo_begin(m, 1, (hipStream_t)stream, &cap);
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("ordering standalone denoises: ") + hipGetErrorString(e));
    Run r{m, (hipStream_t)stream, LaunchCaps{}, &m->aws[0]->scr, m->aws[0].get()};
    const int rc = run_denoise(r, ctx, noise, actions);
    e = solo_end(m, 1, (hipStream_t)stream, cap);
    if (rc == VLA_OK && e != hipSuccess) return fail(VLA_EHIP, std::string("ordering standalone denoises: ") + hipGetErrorString(e));
    return rc;
  })
}

int vla_pipeline_run(vla_model* m, const vla_frame* frames, const float* noise, int32_t R,
                     const vla_sched* sched, float* actions, vla_timing* t) {
  ABI_GUARD({
    if (!m) return fail(VLA_EINVAL, "model is NULL");
    const hipError_t e = solo_drain(m);
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("waiting for standalone calls: ") + hipGetErrorString(e));
    return pipeline_impl(m, frames, noise, R, sched, actions, t);
  })
}

int vla_param_count(const vla_model* m, int32_t* count) {
  ABI_GUARD({
    if (!m || !count) return fail(VLA_EINVAL, "NULL argument");
    *count = (int32_t)m->P.size();
    return VLA_OK;
  })
}

int vla_param_info(const vla_model* m, int32_t i, const char** name, int64_t* numel) {
  ABI_GUARD({
    if (!m || !name || !numel) return fail(VLA_EINVAL, "NULL argument");
    if (i < 0 || i >= (int32_t)m->P.size()) return fail(VLA_EINVAL, "index out of range");
    *name = m->P[i].name.c_str();
    *numel = (int64_t)m->P[i].rows * m->P[i].cols;
    return VLA_OK;
  })
}

int vla_export_param(vla_model* m, const char* name, float* host_dst, int64_t numel) {
  ABI_GUARD({
    if (!m || !name || !host_dst) return fail(VLA_EINVAL, "NULL argument");
    auto it = m->pidx.find(name);
    if (it == m->pidx.end()) return fail(VLA_EINVAL, std::string("no parameter ") + name);
    const ParamRec& p = m->P[it->second];
    if (numel != (int64_t)p.rows * p.cols) return fail(VLA_EINVAL, "numel mismatch");
    const DevTensor& t = m->T[p.tensor];
    std::vector<uint8_t> img(t.bytes());
    HIP_TRY(hipMemcpy(img.data(), m->tptr(p.tensor), img.size(), hipMemcpyDeviceToHost));
    const bool vec = t.vec;
    for (int r = 0; r < p.rows; ++r) {
      const int pr = vec ? 0 : dev_row(p, r);
      for (int col = 0; col < p.cols; ++col) {
        const size_t at = vec ? (size_t)p.row_off + col : t.index(pr, col);
        host_dst[(size_t)r * p.cols + col] = t.dt == DT_BF16 ? bf16_value(((uint16_t*)img.data())[at])
                                                             : ((float*)img.data())[at];
      }
    }
    return VLA_OK;
  })
}

int vla_ctx_export_kv(vla_model* m, const vla_ctx* c, int32_t layer, float* host_k, float* host_v) {
  ABI_GUARD({
    if (!m || !c || !host_k || !host_v) return fail(VLA_EINVAL, "NULL argument");
    if (layer < 0 || layer >= m->c.lm_layers) return fail(VLA_EINVAL, "layer out of range");
    if (c->m != m) return fail(VLA_ESTATE, "context belongs to another model");
    const int P = m->d.prefix, nb = m->d.prefix_pad / 32, hd = m->c.head_dim;
    const int nkv = m->c.lm_kv_heads, kvd = m->d.kvd;
    auto val = [&](const std::vector<uint8_t>& img, size_t i) {
      return m->dt == DT_BF16 ? bf16_value(((const uint16_t*)img.data())[i]) : ((const float*)img.data())[i];
    };
    const size_t nk = ctx_layer_k(m), nv = ctx_layer_v(m);
    std::vector<uint8_t> kimg(nk * m->esz), vimg(nv * m->esz);
    HIP_TRY(hipMemcpy(kimg.data(), (const char*)c->K + layer * nk * m->esz, kimg.size(), hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(vimg.data(), (const char*)c->V + layer * nv * m->esz, vimg.size(), hipMemcpyDeviceToHost));
    for (int p = 0; p < P; ++p)
      for (int j = 0; j < nkv; ++j)
        for (int dd = 0; dd < hd; ++dd) {
          host_k[(size_t)p * kvd + j * hd + dd] = val(kimg, kv_kidx(m->dt, nb, hd, j, p, dd));
          host_v[(size_t)p * kvd + j * hd + dd] = val(vimg, kv_vidx(m->dt, nb, hd, j, p, dd));
        }
    return VLA_OK;
  })
}

int vla_ctx_export_cross(vla_model* m, const vla_ctx* c, int32_t layer, float* host_k, float* host_v) {
  ABI_GUARD({
    if (!m || !c || !host_k || !host_v) return fail(VLA_EINVAL, "NULL argument");
    if (c->m != m) return fail(VLA_ESTATE, "context belongs to another model");
    if (m->c.head != VLA_HEAD_DIT) return fail(VLA_EINVAL, "the model has no DiT head");
    if (layer < 0 || layer >= m->c.ex_layers || layer % 2) return fail(VLA_EINVAL, "layer must be an even DiT layer");
    const int P = m->d.prefix, nb = m->d.prefix_pad / 32, hd = m->d.ehd, nh = m->c.ex_heads;
    const size_t n = cross_elems(m);
    std::vector<uint8_t> kimg(n * m->esz), vimg(n * m->esz);
    const size_t off = (size_t)(layer / 2) * n * m->esz;
    HIP_TRY(hipMemcpy(kimg.data(), (const char*)c->XK + off, kimg.size(), hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(vimg.data(), (const char*)c->XV + off, vimg.size(), hipMemcpyDeviceToHost));
    auto val = [&](const std::vector<uint8_t>& img, size_t i) {
      return m->dt == DT_BF16 ? bf16_value(((const uint16_t*)img.data())[i]) : ((const float*)img.data())[i];
    };
    for (int p = 0; p < P; ++p)
      for (int j = 0; j < nh; ++j)
        for (int dd = 0; dd < hd; ++dd) {
          host_k[(size_t)p * nh * hd + j * hd + dd] = val(kimg, kv_kidx(m->dt, nb, hd, j, p, dd));
          host_v[(size_t)p * nh * hd + j * hd + dd] = val(vimg, kv_vidx(m->dt, nb, hd, j, p, dd));
        }
    return VLA_OK;
  })
}

int vla_ctx_export_cog(vla_model* m, const vla_ctx* c, float* host_dst) {
  ABI_GUARD({
    if (!m || !c || !host_dst) return fail(VLA_EINVAL, "NULL argument");
    if (c->m != m) return fail(VLA_ESTATE, "context belongs to another model");
    if (m->c.head != VLA_HEAD_COG || !c->cog) return fail(VLA_EINVAL, "the model has no cognition-token head");
    HIP_TRY(hipMemcpy(host_dst, c->cog, (size_t)m->c.ex_dim * 4, hipMemcpyDeviceToHost));
    return VLA_OK;
  })
}

int vla_wavelog_enable(vla_model* m, int64_t capacity) {
  ABI_GUARD({
    if (!m) return fail(VLA_EINVAL, "model is NULL");
    if (capacity < 0 || capacity > (int64_t)1 << 30) return fail(VLA_EINVAL, "capacity out of range");
    std::lock_guard<std::mutex> lock(m->mu);
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(wavelog_set(nullptr));
    if (m->wlog) {
      HIP_TRY(hipFree(m->wlog));
      m->wlog = nullptr;
      m->wlog_cap = 0;
    }
    if (capacity == 0) return VLA_OK;
    const size_t per = ((size_t)capacity + WAVELOG_SLICES - 1) / WAVELOG_SLICES;
    const size_t bytes = sizeof(WaveLog) + per * WAVELOG_SLICES * sizeof(WaveRec);
    hipError_t e = hipMalloc(&m->wlog, bytes);
    if (e != hipSuccess) return fail(VLA_ENOMEM, "wave log: hipMalloc failed");
    std::vector<uint8_t> head(offsetof(WaveLog, rec), 0);
    ((WaveLog*)head.data())->cap = (uint32_t)per;
    HIP_TRY(hipMemcpy(m->wlog, head.data(), head.size(), hipMemcpyHostToDevice));
    m->wlog_cap = per;
    HIP_TRY(wavelog_set(m->wlog));
    return VLA_OK;
  })
}

int vla_wavelog_read(vla_model* m, void* host_dst, int64_t max_records, int64_t* n) {
  ABI_GUARD({
    if (!m || !n || (!host_dst && max_records > 0)) return fail(VLA_EINVAL, "NULL argument");
    if (!m->wlog) return fail(VLA_ESTATE, "the wave log is not enabled");
    std::lock_guard<std::mutex> lock(m->mu);
    HIP_TRY(hipDeviceSynchronize());
    std::vector<uint8_t> head(offsetof(WaveLog, rec));
    HIP_TRY(hipMemcpy(head.data(), m->wlog, head.size(), hipMemcpyDeviceToHost));
    WaveLog* h = (WaveLog*)head.data();
    int64_t total = 0, got = 0;
    const int64_t room = std::max<int64_t>(max_records, 0);
    for (int x = 0; x < WAVELOG_SLICES; ++x) {
      const int64_t c = h->count[64 * x];
      total += c;
      const int64_t k = std::min<int64_t>({c, (int64_t)m->wlog_cap, room - got});
      if (k > 0)
        HIP_TRY(hipMemcpy((WaveRec*)host_dst + got, m->wlog->rec + (size_t)x * m->wlog_cap,
                          (size_t)k * sizeof(WaveRec), hipMemcpyDeviceToHost));
      got += std::max<int64_t>(k, 0);
      h->count[64 * x] = 0;
    }
    *n = got;
    if (total > got && room > got) return fail(VLA_ESTATE, "wave log overflowed: raise the capacity");
    HIP_TRY(hipMemcpy(m->wlog, head.data(), head.size(), hipMemcpyHostToDevice));
    return VLA_OK;
  })
}

int vla_debug_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                   const void* W, int32_t ldw, const float* bias, float* C, void* stream) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (M <= 0 || N <= 0 || K <= 0 || K % 8 || lda < K || ldw < K || lda % 8 || ldw % 8)
      return fail(VLA_EINVAL, "shape: M, N, K > 0, K, lda, ldw multiples of 8, lda, ldw >= K");
    if (!A || !W || !C) return fail(VLA_EINVAL, "NULL argument");
    GemmDesc g{dtype == VLA_BF16 ? DT_BF16 : DT_F32, A, lda, W, ldw, M, N, K, Epi()};
    g.epi.kind = EPI_F32;
    g.epi.out = C;
    g.epi.ldo = N;
    g.epi.bias = bias;
    const GemmPlan p = plan_gemm(g);
    Scratch s;
    if (p.scratch_floats) {
      HIP_TRY(hipMalloc(&s.ptr, p.scratch_floats * 4));
      s.floats = p.scratch_floats;
    }
    hipError_t e = launch_gemm(g, s, LaunchCaps{}, (hipStream_t)stream);
    if (s.ptr) {
      hipStreamSynchronize((hipStream_t)stream);
      hipFree(s.ptr);
    }
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("gemm: ") + hipGetErrorString(e));
    return VLA_OK;
  })
}

int vla_gemm_noalloc(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                     const void* W, int32_t ldw, const float* bias, float* C, void* stream) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (M <= 0 || N <= 0 || K <= 0 || K % 8 || lda < K || ldw < K || lda % 8 || ldw % 8)
      return fail(VLA_EINVAL, "shape: M, N, K > 0, K, lda, ldw multiples of 8, lda, ldw >= K");
    if (!A || !W || !C) return fail(VLA_EINVAL, "NULL argument");
    GemmDesc g{dtype == VLA_BF16 ? DT_BF16 : DT_F32, A, lda, W, ldw, M, N, K, Epi()};
    g.epi.kind = EPI_F32;
    g.epi.out = C;
    g.epi.ldo = N;
    g.epi.bias = bias;
    const GemmPlan p = plan_gemm(g);
    if (p.scratch_floats > NOALLOC_SCRATCH_FLOATS)
      return fail(VLA_EUNSUPPORTED, "split-K partials of " + std::to_string(p.scratch_floats) +
                                        " floats exceed the fixed scratch of " +
                                        std::to_string(NOALLOC_SCRATCH_FLOATS) + " floats");
    Scratch s;
    if (p.scratch_floats) {
      VLA_TRY(noalloc_scratch(&s.ptr));
      s.floats = NOALLOC_SCRATCH_FLOATS;
    }
    hipError_t e = launch_gemm(g, s, LaunchCaps{}, (hipStream_t)stream);
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("gemm: ") + hipGetErrorString(e));
    return VLA_OK;
  })
}

int vla_debug_gemm_epi(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, const void* W,
                       const vla_debug_epi* ep, void* stream_) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (!A || !W || !ep) return fail(VLA_EINVAL, "NULL argument");
    const vla_debug_epi& e = *ep;
    if (M <= 0 || N <= 0 || K <= 0 || K % 8) return fail(VLA_EINVAL, "shape: M, N, K > 0, K a multiple of 8");
    if (e.skinny && M > 64) return fail(VLA_EINVAL, "the skinny kernel takes M <= 64");
    const int dt = dtype == VLA_BF16 ? DT_BF16 : DT_F32;
    const size_t esz = dt == DT_BF16 ? 2 : 4;
    hipStream_t st = (hipStream_t)stream_;
    const int kind = e.kind;
    const bool rope = kind == VLA_DEBUG_EPI_QKV_ROPE, qkv = rope || kind == VLA_DEBUG_EPI_QKV_PLAIN;
    if (kind < VLA_DEBUG_EPI_BIAS || kind > VLA_DEBUG_EPI_RESID_NORM) return fail(VLA_EINVAL, "unknown epilogue");
    if (kind == VLA_DEBUG_EPI_GEGLU && N % 32) return fail(VLA_EINVAL, "GEGLU: N must be a multiple of 32");
    if (qkv) {
      if (e.nq < 0 || e.nkv <= 0 || e.hd <= 0 || e.hd % 8 || N != (e.nq + 2 * e.nkv) * e.hd || e.pos0 < 0)
        return fail(VLA_EINVAL, "QKV: N must be (nq + 2 nkv) hd, hd a multiple of 8");
      if (rope && e.hd % 32) return fail(VLA_EINVAL, "QKV_ROPE: hd must be a multiple of 32");
      if (dt == DT_F32 && e.hd > 128) return fail(VLA_EINVAL, "QKV in fp32: hd <= 128");
      if ((e.nq > 0 && !e.q_out) || !e.k_out || !e.v_out) return fail(VLA_EINVAL, "QKV: NULL output");
    } else if (kind == VLA_DEBUG_EPI_STEP) {
      if (!e.x || !e.out) return fail(VLA_EINVAL, "STEP: NULL x or out");
    } else if (kind == VLA_DEBUG_EPI_RESID_NORM) {
      if (!e.resid || !e.gain || !e.out || N > 2048) return fail(VLA_EINVAL, "RESID_NORM: NULL buffer or N > 2048");
    } else if (!e.out) {
      return fail(VLA_EINVAL, "NULL out");
    }
    std::vector<void*> tmp;
    struct Free {
      std::vector<void*>& v;
      ~Free() {
        for (void* p : v) hipFree(p);
      }
    } freer{tmp};
    // temporaries: zeroed and filled by blocking calls; the device is
    // synchronised before the launches on `st`
    auto dalloc = [&](size_t bytes, void** p) -> int {
      HIP_TRY(hipMalloc(p, std::max<size_t>(bytes, 256)));
      tmp.push_back(*p);
      HIP_TRY(hipMemset(*p, 0, std::max<size_t>(bytes, 256)));
      return VLA_OK;
    };
    HIP_TRY(hipStreamSynchronize(st));
    // host images of the operands (logical row-major)
    std::vector<uint8_t> hw((size_t)N * K * esz);
    HIP_TRY(hipMemcpy(hw.data(), W, hw.size(), hipMemcpyDeviceToHost));
    // physical row of logical weight row r: GeGLU gate / up rows interleaved
    // in 16-row blocks; Q and K rows of each head permuted so that RoPE
    // partners (i, i + hd/2) sit 16 columns apart
    const int qk_rows = rope ? (e.nq + e.nkv) * e.hd : 0;
    auto prow = [&](int rr) -> int {
      if (kind == VLA_DEBUG_EPI_GEGLU) {
        const int F = N / 2;
        return rr < F ? 32 * (rr / 16) + rr % 16 : 32 * ((rr - F) / 16) + 16 + (rr - F) % 16;
      }
      if (rope && rr < qk_rows) {
        const int hd = e.hd, half = hd / 2, head = rr / hd, i = rr % hd;
        const int ph = i < half ? 32 * (i / 16) + i % 16 : 32 * ((i - half) / 16) + 16 + (i - half) % 16;
        return head * hd + ph;
      }
      return rr;
    };
    const int fks = (K + frag_slab(dt) - 1) / frag_slab(dt);
    std::vector<uint8_t> pw;
    if (e.skinny) {
      pw.assign((size_t)((N + 31) / 32 * 32) * fks * frag_slab(dt) * esz, 0);
      for (int rr = 0; rr < N; ++rr) {
        const int p = prow(rr);
        for (int k = 0; k < K; ++k)
          std::memcpy(&pw[frag_index(p, k, fks, dt) * esz], &hw[((size_t)rr * K + k) * esz], esz);
      }
    } else {
      pw.assign(hw.size(), 0);
      for (int rr = 0; rr < N; ++rr)
        std::memcpy(&pw[(size_t)prow(rr) * K * esz], &hw[(size_t)rr * K * esz], (size_t)K * esz);
    }
    void* dW = nullptr;
    VLA_TRY(dalloc(pw.size(), &dW));
    HIP_TRY(hipMemcpy(dW, pw.data(), pw.size(), hipMemcpyHostToDevice));
    const void* dA = A;
    if (e.skinny) {  // A in the row-block operand layout
      std::vector<uint8_t> ha((size_t)M * K * esz), pa(afrag_elems(dt, K) * esz, 0);
      HIP_TRY(hipMemcpy(ha.data(), A, ha.size(), hipMemcpyDeviceToHost));
      for (int mm = 0; mm < M; ++mm)
        for (int k = 0; k < K; ++k)
          std::memcpy(&pa[afrag_index(dt, mm, k) * esz], &ha[((size_t)mm * K + k) * esz], esz);
      void* p = nullptr;
      VLA_TRY(dalloc(pa.size(), &p));
      HIP_TRY(hipMemcpy(p, pa.data(), pa.size(), hipMemcpyHostToDevice));
      dA = p;
    }
    Epi x;
    x.afrag = e.skinny ? 1 : 0;
    // operand-type output columns and its device image (row-major, or the
    // row-block operand layout on the skinny path)
    const int ocols = kind == VLA_DEBUG_EPI_GEGLU ? N / 2 : N;
    const bool op_out = kind == VLA_DEBUG_EPI_T || kind == VLA_DEBUG_EPI_GELU || kind == VLA_DEBUG_EPI_SWISH ||
                        kind == VLA_DEBUG_EPI_GEGLU || kind == VLA_DEBUG_EPI_STEP ||
                        kind == VLA_DEBUG_EPI_RESID_NORM;
    const size_t oel = e.skinny ? afrag_elems(dt, ocols) : (size_t)M * ocols;
    void* dout = nullptr;
    if (op_out) VLA_TRY(dalloc(oel * esz, &dout));
    void *dk = nullptr, *dv = nullptr;
    const int kv_nb = (M + 31) / 32;
    float *rc = nullptr, *rs = nullptr;
    switch (kind) {
      case VLA_DEBUG_EPI_BIAS:
        x.kind = EPI_F32;
        x.out = e.out;
        x.ldo = N;
        x.bias = e.bias;
        break;
      case VLA_DEBUG_EPI_T:
      case VLA_DEBUG_EPI_GELU:
      case VLA_DEBUG_EPI_SWISH:
        x.kind = kind == VLA_DEBUG_EPI_T ? EPI_T : kind == VLA_DEBUG_EPI_GELU ? EPI_GELU : EPI_SWISH;
        x.out = dout;
        x.ldo = N;
        x.bias = e.bias;
        break;
      case VLA_DEBUG_EPI_GEGLU:
        x.kind = EPI_GEGLU;
        x.out = dout;
        x.ldo = N / 2;
        break;
      case VLA_DEBUG_EPI_QKV_ROPE:
      case VLA_DEBUG_EPI_QKV_PLAIN: {
        x.kind = rope ? EPI_QKV_ROPE : EPI_QKV_PLAIN;
        x.afrag = 0;
        x.q = e.q_out;
        x.ldq = e.nq * e.hd;
        VLA_TRY(dalloc(kv_kelems(dt, kv_nb, e.hd, e.nkv) * esz, &dk));
        VLA_TRY(dalloc(kv_velems(dt, kv_nb, e.hd, e.nkv) * esz, &dv));
        x.k = dk;
        x.v = dv;
        x.kv_nb = kv_nb;
        x.nq = e.nq;
        x.nkv = e.nkv;
        x.hd = e.hd;
        x.pos0 = e.pos0;
        if (rope) {
          std::vector<float> cs, sn;
          rope_tables(e.pos0 + M, e.hd, cs, sn);
          VLA_TRY(dalloc(cs.size() * 4, (void**)&rc));
          VLA_TRY(dalloc(sn.size() * 4, (void**)&rs));
          HIP_TRY(hipMemcpy(rc, cs.data(), cs.size() * 4, hipMemcpyHostToDevice));
          HIP_TRY(hipMemcpy(rs, sn.data(), sn.size() * 4, hipMemcpyHostToDevice));
          x.rope_cos = rc;
          x.rope_sin = rs;
        }
        break;
      }
      case VLA_DEBUG_EPI_STEP:
        x.kind = EPI_EULER;
        x.bias = e.bias;
        x.x = e.x;
        x.ldx = N;
        x.xop = dout;
        x.ldxop = N;
        x.dt = e.dt;
        x.xs = e.xs;
        break;
      default:  // RESID_NORM: raw split-K partials, summed by the norm
        x.kind = EPI_PART;
        x.afrag = 0;
        break;
    }
    GemmDesc g{dt, dA, K, dW, K, M, N, K, x};
    if (e.skinny) {
      g.frag_ks = fks;
      g.frag_ks0 = 0;
    }
    const GemmPlan p = plan_gemm(g);
    Scratch s;
    if (p.scratch_floats) {
      VLA_TRY(dalloc(p.scratch_floats * 4, (void**)&s.ptr));
      s.floats = p.scratch_floats;
    }
    if (kind == VLA_DEBUG_EPI_RESID_NORM) {
      g.epi.out = s.ptr;
      g.epi.ldo = (int)std::min<size_t>(s.floats, (size_t)INT32_MAX);
    }
    if (e.plan_out) {
      plan_tile(g, p, &e.plan_out[0], &e.plan_out[1]);
      e.plan_out[2] = p.splits;
    }
    HIP_TRY(hipDeviceSynchronize());
    hipError_t err = launch_gemm(g, s, LaunchCaps{}, st);
    if (err != hipSuccess) return fail(VLA_EHIP, std::string("gemm: ") + hipGetErrorString(err));
    if (kind == VLA_DEBUG_EPI_RESID_NORM) {
      NormDesc n;
      n.dtype = dt;
      n.x = e.resid;
      n.ldx = N;
      n.rows = M;
      n.d = N;
      n.part = s.ptr;
      n.splits = p.splits;
      n.g = e.gain;
      n.rms = 1;
      n.out = dout;
      n.ldo = N;
      n.afrag = e.skinny ? 1 : 0;
      err = launch_norm(n, st);
      if (err != hipSuccess) return fail(VLA_EHIP, std::string("norm: ") + hipGetErrorString(err));
    }
    HIP_TRY(hipStreamSynchronize(st));
    // outputs back to the caller's row-major buffers
    if (op_out) {
      std::vector<uint8_t> img(oel * esz), rm((size_t)M * ocols * esz);
      HIP_TRY(hipMemcpy(img.data(), dout, img.size(), hipMemcpyDeviceToHost));
      for (int mm = 0; mm < M; ++mm)
        for (int c = 0; c < ocols; ++c) {
          const size_t at = e.skinny ? afrag_index(dt, mm, c) : (size_t)mm * ocols + c;
          std::memcpy(&rm[((size_t)mm * ocols + c) * esz], &img[at * esz], esz);
        }
      HIP_TRY(hipMemcpy(e.out, rm.data(), rm.size(), hipMemcpyHostToDevice));
    }
    if (qkv) {
      const int kvd = e.nkv * e.hd;
      std::vector<uint8_t> ki(kv_kelems(dt, kv_nb, e.hd, e.nkv) * esz), vi(kv_velems(dt, kv_nb, e.hd, e.nkv) * esz);
      std::vector<uint8_t> kr((size_t)M * kvd * esz), vr((size_t)M * kvd * esz);
      HIP_TRY(hipMemcpy(ki.data(), dk, ki.size(), hipMemcpyDeviceToHost));
      HIP_TRY(hipMemcpy(vi.data(), dv, vi.size(), hipMemcpyDeviceToHost));
      for (int mm = 0; mm < M; ++mm)
        for (int j = 0; j < e.nkv; ++j)
          for (int d = 0; d < e.hd; ++d) {
            const size_t o = ((size_t)mm * kvd + j * e.hd + d) * esz;
            std::memcpy(&kr[o], &ki[kv_kidx(dt, kv_nb, e.hd, j, mm, d) * esz], esz);
            std::memcpy(&vr[o], &vi[kv_vidx(dt, kv_nb, e.hd, j, mm, d) * esz], esz);
          }
      HIP_TRY(hipMemcpy(e.k_out, kr.data(), kr.size(), hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy(e.v_out, vr.data(), vr.size(), hipMemcpyHostToDevice));
    }
    return VLA_OK;
  })
}

int vla_debug_attention(int32_t dtype, int32_t Sq, int32_t nq, int32_t nkv, int32_t hd, const void* q,
                        const void* k0, const void* v0, int32_t S0, const void* k1, const void* v1,
                        int32_t S1, void* out, void* stream) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (Sq <= 0 || nq <= 0 || nkv <= 0 || nq % nkv || hd <= 0 || hd % 8 || hd > 256 || S0 <= 0 ||
        S1 < 0)
      return fail(VLA_EINVAL, "shape");
    if (!q || !k0 || !v0 || !out || (S1 > 0 && (!k1 || !v1))) return fail(VLA_EINVAL, "NULL argument");
    AttnDesc a{};
    a.dtype = dtype == VLA_BF16 ? DT_BF16 : DT_F32;
    a.q = q;
    a.ldq = nq * hd;
    a.k0 = k0;
    a.v0 = v0;
    a.S0 = S0;
    a.k1 = S1 > 0 ? k1 : nullptr;
    a.v1 = S1 > 0 ? v1 : nullptr;
    a.S1 = S1;
    a.ldkv = nkv * hd;
    a.out = out;
    a.ldo = nq * hd;
    a.Sq = Sq;
    a.nq = nq;
    a.nkv = nkv;
    a.hd = hd;
    a.segs = 1;
    const size_t need = attn_scratch_floats(a);
    Scratch s;
    if (need) {
      HIP_TRY(hipMalloc(&s.ptr, need * 4));
      s.floats = need;
    }
    hipError_t e = launch_attention(a, s, LaunchCaps{}, (hipStream_t)stream);
    if (s.ptr) {
      hipStreamSynchronize((hipStream_t)stream);
      hipFree(s.ptr);
    }
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("attention: ") + hipGetErrorString(e));
    return VLA_OK;
  })
}

int vla_debug_norm(int32_t dtype, int32_t rows, int32_t d, float* x, int32_t ldx, const float* part,
                   int32_t splits, const float* bias, const float* colscale, const float* gain,
                   int32_t gain_plus_one, const float* shift, int32_t rms, void* out, int32_t ldo,
                   void* stream) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (rows < 0 || d < 4 || d > 2048 || d % 4 || ldx < d || ldx % 4 || ldo < d || ldo % 4 || splits < 0)
      return fail(VLA_EINVAL, "shape");
    if (rows == 0) return VLA_OK;  // nothing is read or written
    if (!x || !gain || !out || (splits > 0 && !part)) return fail(VLA_EINVAL, "NULL argument");
    NormDesc n{};
    n.dtype = dtype == VLA_BF16 ? DT_BF16 : DT_F32;
    n.x = x;
    n.ldx = ldx;
    n.rows = rows;
    n.d = d;
    n.part = splits > 0 ? part : nullptr;
    n.splits = splits;
    n.bias = bias;
    n.colscale = colscale;
    n.g = gain;
    n.g_plus_one = gain_plus_one ? 1 : 0;
    n.b = shift;
    n.rms = rms ? 1 : 0;
    n.out = out;
    n.ldo = ldo;
    const hipError_t e = launch_norm(n, (hipStream_t)stream);
    if (e == hipErrorInvalidValue) return fail(VLA_EINVAL, "a pointer is not aligned (16 bytes; bf16 out 8)");
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("norm launch: ") + hipGetErrorString(e));
    return VLA_OK;
  })
}

int vla_debug_attention_cache(int32_t dtype, int32_t Sq, int32_t nq, int32_t nkv, int32_t hd,
                              const void* q, const void* k0, const void* v0, int32_t S0, const void* k1,
                              const void* v1, int32_t S1, void* out, void* stream) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (Sq <= 0 || nq <= 0 || nkv <= 0 || nq % nkv || hd <= 0 || hd % 8 || hd > 256 || S0 <= 0 || S1 < 0)
      return fail(VLA_EINVAL, "shape");
    if (dtype == VLA_F32 && hd > 128) return fail(VLA_EINVAL, "fp32 head dim above 128");
    if (!q || !k0 || !v0 || !out || (S1 > 0 && (!k1 || !v1))) return fail(VLA_EINVAL, "NULL argument");
    if (((uintptr_t)out & 15) != 0) return fail(VLA_EINVAL, "out must be 16-byte aligned");
    AttnKvDesc a{};
    a.dtype = dtype == VLA_BF16 ? DT_BF16 : DT_F32;
    a.q = q;
    a.ldq = nq * hd;
    a.k0 = k0;
    a.v0 = v0;
    a.S0 = S0;
    a.k1 = k1;
    a.v1 = v1;
    a.S1 = S1;
    a.out = out;
    a.ldo = nq * hd;
    a.Sq = Sq;
    a.nq = nq;
    a.nkv = nkv;
    a.hd = hd;
    // room for key splits, as the action phases give it (zeroed counters)
    int nc = 0;
    const size_t nf = attn_kv_split_floats(a.dtype, 1, Sq, nq, nkv, hd, S0, S1, &nc);
    void *part = nullptr, *cnt = nullptr;
    if (nf) {
      HIP_TRY(hipMalloc(&part, nf * 4));
      hipError_t ce = hipMalloc(&cnt, (size_t)nc * 4);
      if (ce == hipSuccess) ce = hipMemset(cnt, 0, (size_t)nc * 4);
      if (ce != hipSuccess) {
        hipFree(part);
        hipFree(cnt);
        return fail(VLA_ENOMEM, std::string("attention split room: ") + hipGetErrorString(ce));
      }
      a.part = (float*)part;
      a.part_floats = nf;
      a.cnt = (unsigned*)cnt;
      a.cnt_n = nc;
    }
    hipError_t e = launch_attention_kv(a, LaunchCaps{}, (hipStream_t)stream);
    if (part) {
      hipStreamSynchronize((hipStream_t)stream);
      hipFree(part);
      hipFree(cnt);
    }
    if (e != hipSuccess) return fail(VLA_EHIP, std::string("attention: ") + hipGetErrorString(e));
    return VLA_OK;
  })
}

int vla_kernel_timer(vla_model* m, const char* tag) {
  ABI_GUARD({
    if (!m) return fail(VLA_EINVAL, "model is NULL");
    std::lock_guard<std::mutex> lock(m->mu);
    m->timer_tag = tag ? tag : "";
    m->timer_used = 0;
    return VLA_OK;
  })
}

int vla_kernel_timer_read(vla_model* m, double* total_ms, int64_t* launches) {
  ABI_GUARD({
    if (!m || !total_ms || !launches) return fail(VLA_EINVAL, "NULL argument");
    std::lock_guard<std::mutex> lock(m->mu);
    double tot = 0;
    for (size_t i = 0; i + 1 < m->timer_used; i += 2) {
      HIP_TRY(hipEventSynchronize(m->timer_ev[i + 1]));
      float ms = 0;
      HIP_TRY(hipEventElapsedTime(&ms, m->timer_ev[i], m->timer_ev[i + 1]));
      tot += ms;
    }
    *total_ms = tot;
    *launches = (int64_t)(m->timer_used / 2);
    m->timer_used = 0;
    return VLA_OK;
  })
}

int vla_debug_gemm_plan(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t kind, int32_t skinny,
                        int32_t plan_m, int32_t plan_batch, int32_t* out, int64_t* scratch_floats) {
  ABI_GUARD({
    if (dtype != VLA_F32 && dtype != VLA_BF16) return fail(VLA_EINVAL, "dtype");
    if (!out) return fail(VLA_EINVAL, "out is NULL");
    if (M <= 0 || N <= 0 || K <= 0 || K % 8 || plan_m < 0 || plan_batch < 1)
      return fail(VLA_EINVAL, "shape: M, N, K > 0, K a multiple of 8, plan_m >= 0, plan_batch >= 1");
    if (skinny && M > 64) return fail(VLA_EINVAL, "the skinny kernel takes M <= 64");
    static const int kinds[] = {EPI_F32, EPI_T, EPI_GELU, EPI_SWISH, EPI_GEGLU, EPI_QKV_ROPE, EPI_QKV_PLAIN,
                                EPI_EULER, EPI_PART};
    if (kind < VLA_DEBUG_EPI_BIAS || kind > VLA_DEBUG_EPI_RESID_NORM) return fail(VLA_EINVAL, "unknown epilogue");
    static_assert(VLA_DEBUG_EPI_RESID_NORM - VLA_DEBUG_EPI_BIAS + 1 == sizeof(kinds) / sizeof(kinds[0]),
                  "one internal kind per epilogue");
    const int dt = dtype == VLA_BF16 ? DT_BF16 : DT_F32;
    GemmDesc g{dt, nullptr, K, nullptr, K, M, N, K, Epi()};
    g.epi.kind = kinds[kind - VLA_DEBUG_EPI_BIAS];
    g.plan_m = plan_m;
    g.plan_batch = plan_batch;
    if (skinny) {
      g.frag_ks = (K + frag_slab(dt) - 1) / frag_slab(dt);
      g.epi.afrag = 1;
    }
    const GemmPlan p = plan_gemm(g);
    plan_tile(g, p, &out[0], &out[1]);
    out[2] = p.splits;
    out[3] = p.tiles;
    if (scratch_floats) *scratch_floats = (int64_t)p.scratch_floats;
    return VLA_OK;
  })
}

int vla_debug_generate(uint64_t seed, const char* name, int64_t n, double mean, double stdv,
                       float* host_dst) {
  ABI_GUARD({
    if (!name || !host_dst || n < 0) return fail(VLA_EINVAL, "bad argument");
    gen_normal(seed, name, (size_t)n, mean, stdv, host_dst);
    return VLA_OK;
  })
}

}  // extern "C"
