// gfx950 kernels of the two-phase VLA hot path.
//
// GEMMs and attention run on the matrix cores (MFMA, 64-wide wavefronts):
// bf16 operands use v_mfma_f32_16x16x32_bf16, fp32 operands
// v_mfma_f32_16x16x4_f32; accumulation is always fp32. Norms, softmax,
// activations, RoPE and the Euler update are fp32 and are fused into the
// producing kernel where they are elementwise (GEMM epilogues).
//
// Every reduction has a fixed order that depends only on the problem shape
// (tile sizes, split-K and KV-split factors come from the shape), so results
// do not depend on the grid size, CU mask or on which workgroup ran a tile.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <type_traits>

#include "kernels.h"

namespace vla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NUM_CU_PLAN = 256;  // planner constant; never the live CU count

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
// Residency log (see WaveLog): the log pointer lives in constant memory, so
// the check at the start and at the end of a workgroup is a scalar load that
// issues beside the kernel-argument loads (a vector load there would delay
// every workgroup's first memory round trip); one vector atomic per record
// while logging. No register is held between the two points.
__constant__ WaveLog* g_wavelog = nullptr;

__device__ __forceinline__ void wave_event(uint32_t kind, uint32_t end) {
  WaveLog* L = g_wavelog;
  if (threadIdx.x != 0) return;
  const uint64_t t = wall_clock64();
  const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | 20);  // XCC_ID
  const uint32_t x = xcc & (WAVELOG_SLICES - 1);
  const uint32_t i = atomicAdd(&L->count[64 * x], 1u);
  if (i < L->cap) {
    WaveRec r;
    r.t = t;
    r.hwid = __builtin_amdgcn_s_getreg((31 << 11) | 4);  // HW_ID
    r.xcc = xcc;
    r.kind = kind;
    r.end = end;
    L->rec[(size_t)x * L->cap + i] = r;
  }
}

#define VLA_WAVE_BEGIN(kind)                \
  do {                                      \
    if (g_wavelog) wave_event((kind), 0u);  \
  } while (0)
#define VLA_WAVE_END(kind)                  \
  do {                                      \
    if (g_wavelog) wave_event((kind), 1u);  \
  } while (0)

hipError_t wavelog_set(WaveLog* dev) {
  return hipMemcpyToSymbol(HIP_SYMBOL(g_wavelog), &dev, sizeof(dev));
}

// round to nearest, ties to even (the hardware conversion)
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

// Cross-lane reductions over lanes l ^ 16 and l ^ 32 with the lane-swap
// instructions (no LDS round trip). Both lanes of a pair compute the same
// expression on the same operands, so they hold identical results.
__device__ __forceinline__ float wave_max_x16_x32(float x) {
  const uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t v = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float wave_sum_x16_x32(float x) {
  const uint32_t u = __float_as_uint(x);
  auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t v = __float_as_uint(x);
  auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

template <typename T>
struct TT;
template <>
struct TT<float> {
  static __device__ __forceinline__ float ld(const float* p) { return *p; }
  static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
};
template <>
struct TT<uint16_t> {
  static __device__ __forceinline__ float ld(const uint16_t* p) { return bf2f(*p); }
  static __device__ __forceinline__ void st(uint16_t* p, float v) { *p = f2bf(v); }
};

// x / (1 + e^-z) with the hardware exp2 and reciprocal (about 1 ulp each):
// e^-z = 2^(-z log2 e). For z below about -88 the exponential overflows to
// +inf and the result is -0 or +0, the limit.
__device__ __forceinline__ float x_sigmoid(float x, float z) {
  const float e = __builtin_amdgcn_exp2f(-1.4426950408889634f * z);
  return x * __builtin_amdgcn_rcpf(1.f + e);
}
// GELU, tanh form: 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3);
// since 0.5 (1 + tanh(u)) = 1 / (1 + e^(-2u)) exactly, it is x sigmoid(2u).
__device__ __forceinline__ float gelu_tanh(float x) {
  const float c2 = 1.5957691216057308f;  // 2 sqrt(2 / pi)
  const float x2 = x * x;
  return x_sigmoid(x, c2 * __builtin_fmaf(0.044715f * x2, x, x));
}
__device__ __forceinline__ float swishf(float x) { return x_sigmoid(x, x); }

// One MFMA step over a 16-byte slice of K per lane (8 bf16 or 4 fp32).
__device__ __forceinline__ f32x4 mfma_step(uint4 a, uint4 b, f32x4 c, uint16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_step(uint4 a, uint4 b, f32x4 c, float) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  return c;
}

// Masked loads go through buffer resources: a byte offset at or past the
// resource's range returns zero in hardware, so a masked lane just gets an
// out-of-range offset and no branch is needed. (A predicated pointer load
// would become a branch, and the compiler drains every outstanding load at
// such joins, which serialises memory traffic.)
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr uint32_t OOB = 0x80000000u;

__device__ __forceinline__ Rsrc rsrc(const void* base, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0,
                                           (int)(bytes < 0x7FFFFFFFu ? bytes : 0x7FFFFFFFu), 0x00020000);
}
// bytes spanned by `rows` rows of `len` elements at row stride `ld`
__device__ __forceinline__ size_t span(int rows, size_t ld, int len, size_t esz) {
  return rows > 0 ? ((size_t)(rows - 1) * ld + len) * esz : 0;
}
__device__ __forceinline__ uint4 bld16(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// the same with a wave-uniform byte offset added (in a scalar register)
__device__ __forceinline__ uint4 bld16s(Rsrc r, uint32_t off, uint32_t soff) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0));
}
// 16 bytes per lane from the buffer straight into the LDS: lane l writes
// bytes [16 l, 16 l + 16) after `dst` (which must be the same in every lane);
// an out-of-range lane writes zeros
__device__ __forceinline__ void bld16_lds(Rsrc r, void* dst, uint32_t off, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16, off, soff, 0, 0);
}
// s_waitcnt operand that waits for every outstanding vector memory load
// (vmcnt 0; expcnt and lgkmcnt left at their maxima)
constexpr int VMCNT0 = 0x0F70;
__device__ __forceinline__ float bld1(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
// Loads and stores with the sc1 cache policy (the one agent-scope atomic
// loads and stores get): stores write through to the memory side and loads
// are served from it, so data one workgroup writes is seen by a workgroup on
// another XCD, whose L2 is a different cache.
constexpr int CP_SC1 = 16;
__device__ __forceinline__ f32x4 bld16_sc1(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, CP_SC1));
}
__device__ __forceinline__ float bld1_sc1(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, CP_SC1));
}
__device__ __forceinline__ void bst16_sc1(Rsrc r, uint32_t off, f32x4 v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, CP_SC1);
}
__device__ __forceinline__ void bst1_sc1(Rsrc r, uint32_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, off, 0, CP_SC1);
}
__device__ __forceinline__ f32x4 bld4f(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// ---------------------------------------------------------------------------
// GEMM epilogues
// ---------------------------------------------------------------------------

// Index of output element (m, n) of an operand-type epilogue output.
template <typename T>
__device__ __forceinline__ size_t out_at(const Epi& e, int m, int n, int ld, size_t blk) {
  constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
  return e.afrag ? afrag_index_blk(DT, m, n, e.blk_rows, blk) : (size_t)m * ld + n;
}
// key index and element offset of row m's own K / V (frame blocks)
__device__ __forceinline__ int epi_key(const Epi& e, int m) { return e.blk_rows > 0 ? m % e.blk_rows : m; }
__device__ __forceinline__ size_t epi_kblk(const Epi& e, int m, size_t blk) {
  return e.blk_rows > 0 ? (size_t)(m / e.blk_rows) * blk : 0;
}

// KIND >= 0 fixes the epilogue kind at compile time (only that kind's code is
// emitted); KIND = -1 dispatches on e.kind at run time.
template <typename T, int KIND = -1>
__device__ __forceinline__ void epi_one(const Epi& e, int m, int n, float v) {
  switch (KIND >= 0 ? KIND : e.kind) {
    case EPI_F32: {
      if (e.bias) v += e.bias[n];
      if (e.rowadd) v += e.rowadd[(size_t)(m % e.rowadd_period) * e.ldra + n];
      ((float*)e.out)[(size_t)m * e.ldo + n] = v;
      break;
    }
    case EPI_T: {
      if (e.bias) v += e.bias[n];
      TT<T>::st((T*)e.out + out_at<T>(e, m, n, e.ldo, e.blk_out), v);
      break;
    }
    case EPI_RESID: {
      if (e.bias) v += e.bias[n];
      e.resid[(size_t)m * e.ldr + n] += v;
      break;
    }
    case EPI_GELU: {
      if (e.bias) v += e.bias[n];
      TT<T>::st((T*)e.out + out_at<T>(e, m, n, e.ldo, e.blk_out), gelu_tanh(v));
      break;
    }
    case EPI_SWISH: {
      if (e.bias) v += e.bias[n];
      TT<T>::st((T*)e.out + out_at<T>(e, m, n, e.ldo, e.blk_out), swishf(v));
      break;
    }
    case EPI_QKV_PLAIN: {
      constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
      const int qcols = e.nq * e.hd, kcols = e.nkv * e.hd;
      if (n < qcols) {
        TT<T>::st((T*)e.q + (size_t)m * e.ldq + n, v);
      } else if (n < qcols + kcols) {
        const int c = n - qcols;
        TT<T>::st((T*)e.k + epi_kblk(e, m, e.blk_k) + kv_kidx(DT, e.kv_nb, e.hd, c / e.hd, epi_key(e, m), c % e.hd), v);
      } else {
        const int c = n - qcols - kcols;
        TT<T>::st((T*)e.v + epi_kblk(e, m, e.blk_v) + kv_vidx(DT, e.kv_nb, e.hd, c / e.hd, epi_key(e, m), c % e.hd), v);
      }
      break;
    }
    case EPI_EULER: {
      if (e.bias) v += e.bias[n];
      float* xp = e.x + (size_t)m * e.ldx + n;
      const float xn = __builtin_fmaf(e.dt, v, *xp * e.xs);
      *xp = xn;
      TT<T>::st((T*)e.xop + out_at<T>(e, m, n, e.ldxop, e.blk_xop), xn);
      break;
    }
    default:
      break;
  }
}

// n: a physical column with n % 32 < 16; v1 is the value of column n + 16.
template <typename T, int KIND = -1>
__device__ __forceinline__ void epi_pair(const Epi& e, int M, int N, int m, int n, float v0,
                                         float v1) {
  const int kind = KIND >= 0 ? KIND : e.kind;
  if (m >= M) return;
  if (kind == EPI_GEGLU) {
    if (n + 16 >= N) return;
    const int g = n >> 5, j = n & 15;
    TT<T>::st((T*)e.out + out_at<T>(e, m, 16 * g + j, e.ldo, e.blk_out), gelu_tanh(v0) * v1);
    return;
  }
  if (kind == EPI_QKV_ROPE) {
    if (n + 16 >= N) return;
    const int hd = e.hd, qcols = e.nq * hd, kcols = e.nkv * hd;
    if (n < qcols + kcols) {
      const bool isq = n < qcols;
      const int rn = isq ? n : n - qcols;
      const int head = rn / hd, p = rn - head * hd;
      const int i = 16 * (p >> 5) + (p & 15);  // rotate-half pair (i, i + hd/2)
      const int key = epi_key(e, m);
      const size_t t = (size_t)(e.pos0 + key) * (hd / 2) + i;
      const float c = e.rope_cos[t], s = e.rope_sin[t];
      if (isq) {
        T* dst = (T*)e.q + (size_t)m * e.ldq + head * hd;
        TT<T>::st(dst + i, v0 * c - v1 * s);
        TT<T>::st(dst + i + hd / 2, v1 * c + v0 * s);
      } else {
        constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
        T* dst = (T*)e.k + epi_kblk(e, m, e.blk_k);
        TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, i), v0 * c - v1 * s);
        TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, i + hd / 2), v1 * c + v0 * s);
      }
    } else {
      constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
      const int c0 = n - qcols - kcols, c1 = c0 + 16, key = epi_key(e, m);
      T* dst = (T*)e.v + epi_kblk(e, m, e.blk_v);
      TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, c0 / hd, key, c0 % hd), v0);
      TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, c1 / hd, key, c1 % hd), v1);
    }
    return;
  }
  if (n < N) epi_one<T, KIND>(e, m, n, v0);
  if (n + 16 < N) epi_one<T, KIND>(e, m, n + 16, v1);
}

// The epilogue of PER column pairs of one thread (pair k: row m[k], columns
// n[k] and n[k] + 16, values v0[k], v1[k]), with the arithmetic of epi_pair
// on each pair. Everything the epilogue reads (bias, rowadd, Euler state,
// RoPE tables) is loaded for all pairs before the first store: the vector
// memory counter keeps loads and stores in one issue order, so a load placed
// after a store waits for that store's write to complete, and one epi_pair
// after another would serialise on them. Rows m[k] >= M are skipped.
template <typename T, int PER, int KIND = -1>
__device__ __forceinline__ void epi_pairs(const Epi& e, int M, int N, const int (&m)[PER],
                                          const int (&n)[PER], float (&v0)[PER], float (&v1)[PER]) {
  const int kind = KIND >= 0 ? KIND : e.kind;
  const bool biased = kind == EPI_F32 || kind == EPI_T || kind == EPI_RESID || kind == EPI_GELU ||
                      kind == EPI_SWISH || kind == EPI_EULER;
  if (biased && e.bias) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (n[k] < N) v0[k] += e.bias[n[k]];
      if (n[k] + 16 < N) v1[k] += e.bias[n[k] + 16];
    }
  }
  if (kind == EPI_F32 && e.rowadd) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (m[k] >= M) continue;
      const float* ra = e.rowadd + (size_t)(m[k] % e.rowadd_period) * e.ldra;
      if (n[k] < N) v0[k] += ra[n[k]];
      if (n[k] + 16 < N) v1[k] += ra[n[k] + 16];
    }
  }
  if (kind == EPI_RESID || kind == EPI_EULER) {
    // read-modify-write operands: the residual stream, or the Euler state x
    float* base = kind == EPI_RESID ? e.resid : e.x;
    const int ld = kind == EPI_RESID ? e.ldr : e.ldx;
    float r0[PER], r1[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const bool ok = m[k] < M;
      r0[k] = ok && n[k] < N ? base[(size_t)m[k] * ld + n[k]] : 0.f;
      r1[k] = ok && n[k] + 16 < N ? base[(size_t)m[k] * ld + n[k] + 16] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (m[k] >= M) continue;
      float* p = base + (size_t)m[k] * ld + n[k];
      if (kind == EPI_RESID) {
        if (n[k] < N) p[0] = r0[k] + v0[k];
        if (n[k] + 16 < N) p[16] = r1[k] + v1[k];
      } else {
        if (n[k] < N) {
          const float xn = __builtin_fmaf(e.dt, v0[k], r0[k] * e.xs);
          p[0] = xn;
          TT<T>::st((T*)e.xop + out_at<T>(e, m[k], n[k], e.ldxop, e.blk_xop), xn);
        }
        if (n[k] + 16 < N) {
          const float xn = __builtin_fmaf(e.dt, v1[k], r1[k] * e.xs);
          p[16] = xn;
          TT<T>::st((T*)e.xop + out_at<T>(e, m[k], n[k] + 16, e.ldxop, e.blk_xop), xn);
        }
      }
    }
    return;
  }
  if (kind == EPI_QKV_ROPE) {
    const int hd = e.hd, qcols = e.nq * hd, kcols = e.nkv * hd;
    float c[PER], sn[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      c[k] = 1.f;
      sn[k] = 0.f;
      if (m[k] < M && n[k] + 16 < N && n[k] < qcols + kcols) {
        const int rn = n[k] < qcols ? n[k] : n[k] - qcols;
        const int pp = rn % hd;
        const int i = 16 * (pp >> 5) + (pp & 15);
        const size_t t = (size_t)(e.pos0 + epi_key(e, m[k])) * (hd / 2) + i;
        c[k] = e.rope_cos[t];
        sn[k] = e.rope_sin[t];
      }
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (m[k] >= M || n[k] + 16 >= N) continue;
      if (n[k] < qcols + kcols) {
        const bool isq = n[k] < qcols;
        const int rn = isq ? n[k] : n[k] - qcols;
        const int head = rn / hd, pp = rn - head * hd;
        const int i = 16 * (pp >> 5) + (pp & 15);
        const float a = v0[k] * c[k] - v1[k] * sn[k], b = v1[k] * c[k] + v0[k] * sn[k];
        if (isq) {
          T* dst = (T*)e.q + (size_t)m[k] * e.ldq + head * hd;
          TT<T>::st(dst + i, a);
          TT<T>::st(dst + i + hd / 2, b);
        } else {
          constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
          const int key = epi_key(e, m[k]);
          T* dst = (T*)e.k + epi_kblk(e, m[k], e.blk_k);
          TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, i), a);
          TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, i + hd / 2), b);
        }
      } else {
        epi_pair<T, KIND>(e, M, N, m[k], n[k], v0[k], v1[k]);  // V columns: stores only
      }
    }
    return;
  }
  // the rest only store: bias and rowadd are already in v0 / v1
  Epi f = e;
  f.bias = nullptr;
  f.rowadd = nullptr;
#pragma unroll
  for (int k = 0; k < PER; ++k) epi_pair<T, KIND>(f, M, N, m[k], n[k], v0[k], v1[k]);
}

// ---------------------------------------------------------------------------
// GEMM: C[M, N] = A[M, K] W[N, K]^T, both operands K-contiguous.
// 256 threads = 4 waves in a 2 x 2 arrangement; each wave owns a
// (BM/2) x (BN/2) block of 16 x 16 MFMA tiles. A and W tiles go through a
// two-stage LDS ring (rows padded against bank conflicts) fed by a ring of PD
// K-tiles held in registers, one barrier per K-step. The accumulators are
// staged through LDS for the epilogue, so epilogue stores are row-contiguous.
// With split-K each split writes its raw fp32 partial ([split][M][N]); a
// second kernel sums the partials in split order and applies the epilogue, so
// the result does not depend on which split finishes first. Tiles are visited
// grid-stride so a capped grid computes the same tiles.
// ---------------------------------------------------------------------------

#ifndef VLA_GEMM_LDS_PAD
#define VLA_GEMM_LDS_PAD 2  // LDS row padding of the GEMM tiles, in 16-byte units (32 B: fewest bank conflicts measured)
#endif

// Compile-time loop: f(integral_constant<int, I>) for I = B .. E-1, so that
// register arrays are indexed by constants even where the loop body is too
// large for the unroller.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

template <typename T, int BM, int BN, int BK, int WGM, int PAD = VLA_GEMM_LDS_PAD>
struct GemmSmem {
  static constexpr int VEC = 16 / sizeof(T);
  static constexpr int LDS = BK + VEC * PAD;
  static constexpr int CLD = BN + 4;
  union {
    struct {
      T a[2][BM * LDS];
      T b[2][BN * LDS];
    } ld;
    float c[WGM * 16 * CLD];  // one 16-row slice of every wave row
  };
};
// Direct-load variant: stage 0 of the operand ring shares this object with the
// epilogue slice; stage 1 is a separate __shared__ array, so the compiler can
// tell the two stages apart and lets the LDS reads of one stage run while
// loads into the other are in flight.
template <typename T, int BM, int BN, int BK, int WGM>
struct GemmSmemDL {
  static constexpr int CLD = BN + 4;
  union {
    T d[(BM + BN) * BK];
    float c[WGM * 16 * CLD];
  };
};

// Waves per SIMD each tile is built for, so that its registers leave room
// for the workgroups its LDS allows on a CU (160 KB): the 4-wave 128 x 128
// bf16 tile (80 KB) two per CU, the smaller 4-wave bf16 tiles (40 and 30 KB)
// four (the fp32 tiles, which only the small test models run, three); the
// 8-wave 256 x 256 tile runs alone. Without it the compiler may take a few
// registers more than that leaves (the 128 x 128 GeGLU tile took 260 of
// 256) and a CU then holds one workgroup fewer.
constexpr int gemm_waves_per_eu(int bm, int waves, bool dl, int esize) {
  return dl || waves != 4 ? 2 : esize == 4 ? 3 : bm >= 128 ? 2 : 4;
}

// KIND >= 0: the epilogue kind fixed at compile time (the tiles of the
// batched action loops, short launches whose code should stay in the
// instruction cache); KIND = -1: chosen at run time from e.kind.
template <typename T, int BM, int BN, int BK, int WGM = 2, int WGN = 2, int PD = 1, int PAD = VLA_GEMM_LDS_PAD,
          bool DL = false, int KIND = -1>
__global__ __launch_bounds__(64 * WGM * WGN)
__attribute__((amdgpu_waves_per_eu(gemm_waves_per_eu(BM, WGM * WGN, DL, (int)sizeof(T))))) void k_gemm(const T* __restrict__ A, int lda,
                                              const T* __restrict__ W, int ldw, int M, int N,
                                              int K, int kchunk, int splits, int tiles_m,
                                              int tiles_n, int group_m, Epi e, float* __restrict__ part) {
  VLA_WAVE_BEGIN(KK_GEMM);
  using SM = std::conditional_t<DL, GemmSmemDL<T, BM, BN, BK, WGM>, GemmSmem<T, BM, BN, BK, WGM, PAD>>;
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SW = 4 * VEC;  // K covered by one MFMA step across the 4 lane groups
  constexpr int LDS = BK + VEC * PAD;
  constexpr int CLD = SM::CLD;
  constexpr int NT = 64 * WGM * WGN;  // threads: a WGM x WGN grid of waves
  constexpr int WM = BM / WGM, WN = BN / WGN, TM = WM / 16, TN = WN / 16;
  constexpr int KV = BK / VEC;
  constexpr int AV = BM * KV / NT, BV = BN * KV / NT;
  static_assert(AV >= 1 && BV >= 1 && (BM * KV) % NT == 0 && (BN * KV) % NT == 0, "tile");
  static_assert(WM % 16 == 0 && WN % 16 == 0, "wave tile");
  static_assert(BN % 32 == 0, "paired epilogues need 32-column groups");
  __shared__ __attribute__((aligned(16))) SM sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int ntiles = tiles_m * tiles_n * splits;
  const T dummy = T();
  const Rsrc ra_r = rsrc(A, span(M, lda, K, sizeof(T)));
  const Rsrc rb_r = rsrc(W, span(N, ldw, K, sizeof(T)));

  // Workgroups are dispatched round-robin over the 8 XCDs (workgroup b on
  // XCD b % 8), each with its own L2. Giving every XCD a contiguous range of
  // tiles keeps the row tiles that share a weight block (consecutive tile
  // indices) on one XCD, so the block comes from HBM once. Any bijection of
  // the workgroup index gives the same results.
  // GeGLU of the direct-load tile into row-major bf16: formed in registers
  // (see below); uniform over the launch
  const int ekind = KIND >= 0 ? KIND : e.kind;
  const bool reg_geglu = DL && sizeof(T) == 2 && splits == 1 && ekind == EPI_GEGLU && !e.afrag &&
                         e.blk_rows == 0 && (((uintptr_t)e.out & 15) == 0) && e.ldo % 8 == 0;
  const int G = gridDim.x;
  const int first = G % 8 == 0 ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8) : (int)blockIdx.x;
  const int plane = tiles_m * tiles_n;
  for (int tile = first; tile < ntiles; tile += G) {
    // K split slowest. Within a split, bands of group_m row tiles in turn;
    // inside a band the row tile is fastest, then the column tile. The ~32
    // tiles an XCD runs at once then share group_m row tiles of A and a few
    // column tiles of W in its L2 (group_m = tiles_m, one band, when all of
    // A fits in L2: each weight block is then read once per XCD).
    const int s = tile / plane, r = tile % plane;
    const int band = r / (group_m * tiles_n), tm0 = band * group_m;
    const int gm = min(group_m, tiles_m - tm0), q = r - band * group_m * tiles_n;
    const int tm = tm0 + q % gm, tn = q / gm;
    const int m0 = tm * BM, n0 = tn * BN;
    const int kbeg = s * kchunk, kend = min(K, kbeg + kchunk);
    const int nk = (kend - kbeg + BK - 1) / BK;

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    if constexpr (DL) {
      // Operands go from global memory straight into LDS (buffer loads with
      // the LDS as destination: each wave instruction writes 1 KB, lane l at
      // byte 16 l), two stages. A K-tile row is BK elements = 8 chunks of 16
      // bytes with no padding; chunk c of tile row r sits at chunk position
      // c ^ (r % 8), so the 16-byte fragment reads of 8 consecutive rows hit
      // distinct banks. Lane l of an instruction covering rows 8g .. 8g + 7
      // loads row 8g + l / 8, chunk (l % 8) ^ (l / 8): each row is still read
      // as one contiguous 128-byte line. Out-of-range rows and chunks read as
      // zero through the buffer range check.
      static_assert(sizeof(T) == 2 && BK / VEC == 8, "direct loads: 8 chunks per tile row");
      static_assert((BM / 8) % (NT / 64) == 0 && (BN / 8) % (NT / 64) == 0, "direct loads per wave");
      __shared__ __attribute__((aligned(16))) T d1[(BM + BN) * BK];
      constexpr int LA = BM / 8 / (NT / 64), LB = BN / 8 / (NT / 64);  // instructions per wave
      const int lr = lane >> 3, lcol = ((lane & 7) ^ lr) * VEC;
      uint32_t aoff[LA], boff[LB];
#pragma unroll
      for (int i = 0; i < LA; ++i) {
        const int gm = m0 + (wave * LA + i) * 8 + lr;
        aoff[i] = gm < M ? (uint32_t)(((size_t)gm * lda + lcol) * sizeof(T)) : OOB;
      }
#pragma unroll
      for (int i = 0; i < LB; ++i) {
        const int gn = n0 + (wave * LB + i) * 8 + lr;
        boff[i] = gn < N ? (uint32_t)(((size_t)gn * ldw + lcol) * sizeof(T)) : OOB;
      }
      auto issue = [&](T* d, int k0) {
        const bool kok = lcol < kend - k0;
        const uint32_t soff = (uint32_t)k0 * sizeof(T);
#pragma unroll
        for (int i = 0; i < LA; ++i)
          bld16_lds(ra_r, d + (wave * LA + i) * 8 * BK, kok ? aoff[i] : OOB, soff);
#pragma unroll
        for (int i = 0; i < LB; ++i)
          bld16_lds(rb_r, d + (BM + (wave * LB + i) * 8) * BK, kok ? boff[i] : OOB, soff);
      };
      // fragment reads: tile row (lane % 16) + 16 i of the wave's rows, chunk
      // 4 ks + lane / 16, at chunk position chunk ^ (lane % 8)
      const int fr = lane & 15, fp = ((lane >> 4) ^ (lane & 7)) * VEC;
      auto compute_dl = [&](const T* d) {
        const T* sa = d + (wm * WM + fr) * BK;
        const T* sb = d + (BM + wn * WN + fr) * BK;
#pragma unroll
        for (int ks = 0; ks < BK / SW; ++ks) {
          const int cp = fp ^ (ks * 4 * VEC);
          uint4 af[TM], bfg[TN];
#pragma unroll
          for (int j = 0; j < TN; ++j) bfg[j] = *(const uint4*)(sb + j * 16 * BK + cp);
#pragma unroll
          for (int i = 0; i < TM; ++i) af[i] = *(const uint4*)(sa + i * 16 * BK + cp);
          // all fragment reads of the K-slab go out before its first MFMA
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_step(af[i], bfg[j], acc[i][j], dummy);
        }
      };
      // step: request the next K-tile into the other stage, multiply this
      // one, wait for this wave's loads, one barrier
      T* d0 = sm.d;
      __syncthreads();  // the previous tile's epilogue is done with the LDS
      issue(d0, kbeg);
      __builtin_amdgcn_s_waitcnt(VMCNT0);
      __syncthreads();  // tile 0 is in LDS
      for (int it = 0; it < nk; it += 2) {
        if (it + 1 < nk) issue(d1, kbeg + (it + 1) * BK);
        compute_dl(d0);
        __builtin_amdgcn_s_waitcnt(VMCNT0);
        __syncthreads();
        if (it + 1 < nk) {
          if (it + 2 < nk) issue(d0, kbeg + (it + 2) * BK);
          compute_dl(d1);
          __builtin_amdgcn_s_waitcnt(VMCNT0);
          __syncthreads();
        }
      }
      // GeGLU straight from the accumulators: gate column n (n % 32 < 16)
      // and its up column n + 16 sit in tiles j = 2g and 2g + 1 of the same
      // lane, so each lane forms its outputs in registers. The bf16 tile
      // (BM x BN/2) is staged once in LDS, wave row 0 in stage 0 and wave
      // row 1 in stage 1 (rows padded to OLD elements, so the four row
      // groups of one store hit different banks), then every thread stores
      // 16-byte runs of 8 output columns. After the K loop's last barrier
      // no stage is read any more.
      if (reg_geglu) {
        constexpr int OLD = BN / 2 + 8;
        static_assert(WGM == 2 && BM / 2 * OLD <= (BM + BN) * BK, "staging fits a stage");
        static_assert(TN % 2 == 0, "gate / up tiles in one wave");
        uint16_t* ob = (uint16_t*)(wm == 0 ? d0 : d1);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int g = 0; g < TN / 2; ++g)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int lrow = i * 16 + (lane >> 4) * 4 + r;
              const int ocol = wn * (WN / 2) + 16 * g + (lane & 15);
              ob[lrow * OLD + ocol] = f2bf(gelu_tanh(acc[i][2 * g][r]) * acc[i][2 * g + 1][r]);
            }
        __syncthreads();
        constexpr int CPR = BN / 16;  // 16-byte chunks per output row
        const int ncols = N / 2, c00 = n0 / 2;
#pragma unroll
        for (int k = 0; k < BM * CPR / NT; ++k) {
          const int q = tid + k * NT, row = q / CPR, c = q % CPR;
          const int m = m0 + row;
          const int col0 = c00 + c * 8;
          if (m >= M || col0 >= ncols) continue;
          const uint16_t* src = (const uint16_t*)(row < BM / 2 ? d0 : d1) + (row % (BM / 2)) * OLD + c * 8;
          uint16_t* dst = (uint16_t*)e.out + (size_t)m * e.ldo + col0;
          if (col0 + 8 <= ncols) {
            *(uint4*)dst = *(const uint4*)src;
          } else {
            for (int t = 0; t < ncols - col0; ++t) dst[t] = src[t];
          }
        }
      }
    } else {
      auto compute = [&](int buf) {
        const T* sa = sm.ld.a[buf];
        const T* sb = sm.ld.b[buf];
#pragma unroll
        for (int ks = 0; ks < BK / SW; ++ks) {
          uint4 af[TM], bfg[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i)
            af[i] = *(const uint4*)(sa + (wm * WM + i * 16 + (lane & 15)) * LDS + ks * SW +
                                    (lane >> 4) * VEC);
#pragma unroll
          for (int j = 0; j < TN; ++j)
            bfg[j] = *(const uint4*)(sb + (wn * WN + j * 16 + (lane & 15)) * LDS + ks * SW +
                                     (lane >> 4) * VEC);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_step(af[i], bfg[j], acc[i][j], dummy);
        }
      };

      // K-tiles it+1 .. it+PD are in registers (ring of PD buffers) while tile
      // it is multiplied from LDS; the loop is unrolled by PD so every buffer
      // index is a compile-time constant.
      uint4 ra[PD][AV], rb[PD][BV];
      // Per-thread load offsets, fixed for the tile: thread tid loads the
      // 16-byte column slice kc of rows (tid + i NT) / KV (NT is a multiple of
      // KV, so kc is the same for every i). Each K-step then adds the uniform
      // k0 as the scalar offset; rows past M / N and columns past kend read as
      // zero (out-of-range buffer offset).
      const int kc = (tid % KV) * VEC;
      uint32_t aoff[AV], boff[BV];
#pragma unroll
      for (int i = 0; i < AV; ++i) {
        const int gm = m0 + (tid + i * NT) / KV;
        aoff[i] = gm < M ? (uint32_t)(((size_t)gm * lda + kc) * sizeof(T)) : OOB;
      }
#pragma unroll
      for (int i = 0; i < BV; ++i) {
        const int gn = n0 + (tid + i * NT) / KV;
        boff[i] = gn < N ? (uint32_t)(((size_t)gn * ldw + kc) * sizeof(T)) : OOB;
      }
      auto gload = [&](int k0, uint4 (&xa)[AV], uint4 (&xb)[BV]) {
        const bool kok = kc < kend - k0;  // this thread's slice lies before kend
        const uint32_t soff = (uint32_t)k0 * sizeof(T);
#pragma unroll
        for (int i = 0; i < AV; ++i) xa[i] = bld16s(ra_r, kok ? aoff[i] : OOB, soff);
#pragma unroll
        for (int i = 0; i < BV; ++i) xb[i] = bld16s(rb_r, kok ? boff[i] : OOB, soff);
      };
      auto sstore = [&](int buf, const uint4 (&xa)[AV], const uint4 (&xb)[BV]) {
#pragma unroll
        for (int i = 0; i < AV; ++i) {
          const int c = tid + i * NT, r = c / KV, kc = (c % KV) * VEC;
          *(uint4*)(sm.ld.a[buf] + r * LDS + kc) = xa[i];
        }
#pragma unroll
        for (int i = 0; i < BV; ++i) {
          const int c = tid + i * NT, r = c / KV, kc = (c % KV) * VEC;
          *(uint4*)(sm.ld.b[buf] + r * LDS + kc) = xb[i];
        }
      };
      // iteration it: tile it is multiplied from LDS buffer it & 1 (its MFMAs
      // run while the wave goes on), tile it+1 (ring slot (it+1) % PD) goes to
      // the other buffer, tile it+1+PD is requested into the freed slot, then
      // one barrier. Loads and stores are issued unconditionally (tiles past
      // the end read as zero through the buffer range check), so every path has
      // the same loads in flight and each wait covers only the oldest ring slot.
      auto step = [&](int it, uint4 (&xa)[AV], uint4 (&xb)[BV]) {
        if (it < nk) compute(it & 1);
        sstore((it + 1) & 1, xa, xb);
        gload(kbeg + (it + 1 + PD) * BK, xa, xb);
        __syncthreads();
      };

      __syncthreads();  // the previous tile's epilogue is done with the LDS
      gload(kbeg, ra[0], rb[0]);
      sstore(0, ra[0], rb[0]);
      // the ring slots must be requested in the order the loop consumes them:
      // the scheduler may not interleave them
#pragma unroll
      for (int q = 0; q < PD; ++q) {
        gload(kbeg + (1 + q) * BK, ra[(1 + q) % PD], rb[(1 + q) % PD]);
        __builtin_amdgcn_sched_barrier(0);
      }
      __syncthreads();  // tile 0 is in LDS
      for (int it = 0; it < nk; it += PD) {
#pragma unroll
        for (int q = 0; q < PD; ++q) step(it + q, ra[(q + 1) % PD], rb[(q + 1) % PD]);
      }

    }

    if (reg_geglu) continue;  // stored above
    // epilogue in 16-row slices: slice i of every wave row goes through LDS,
    // then all threads apply the epilogue with row-contiguous stores
    float* P = (ekind == EPI_PART ? (float*)e.out : part) + (size_t)s * M * N;
    const bool direct = splits == 1 && ekind != EPI_PART;
    // In the direct epilogue thread tid always owns the same two columns,
    // na and na + 16 (pair index tid % (BN / 2), since NT is a multiple of
    // BN / 2). Epilogues that only store, or that read nothing but the bias,
    // take a short path: the bias is loaded once per tile, and each slice's
    // stores go out back to back. (A load issued between stores would wait
    // for all of them: the vector memory counter keeps loads and stores in
    // one issue order.)
    static_assert(NT % (BN / 2) == 0, "fixed columns per thread");
    const int qc = tid % (BN / 2), colc = (qc >> 4) * 32 + (qc & 15);
    const int na = n0 + colc, nb = na + 16;
    const int ek = ekind;
    // (the row-operand paths are left out of the largest tile, whose 128
    // accumulators per thread leave few registers; it runs the FFN GEMMs)
    constexpr bool ROWK = TM * TN < 32;
    const bool fast = direct && (ek == EPI_GEGLU || ek == EPI_T || ek == EPI_GELU || ek == EPI_SWISH ||
                                 (ek == EPI_F32 && !e.rowadd) ||
                                 (ROWK && (ek == EPI_QKV_ROPE || ek == EPI_QKV_PLAIN || ek == EPI_EULER)));
    const bool hasb = fast && ek != EPI_GEGLU && ek != EPI_QKV_ROPE && ek != EPI_QKV_PLAIN && e.bias;
    float ba = 0.f, bb = 0.f;
    if (hasb) {
      if (na < N) ba = e.bias[na];
      if (nb < N) bb = e.bias[nb];
    }
    // Row-major operand-type outputs of GeGLU, store, GELU and swish take
    // 8 consecutive output columns per thread and row: one 16-byte store
    // (two for fp32) instead of eight element stores. Thread tid always owns
    // the same 8-column chunk (NT is a multiple of the chunks per row), so
    // its bias is loaded once per tile.
    const bool geglu = ek == EPI_GEGLU;
    const bool vec8 = fast && !e.afrag && e.blk_rows == 0 &&
                      (geglu || ek == EPI_T || ek == EPI_GELU || ek == EPI_SWISH) &&
                      (((uintptr_t)e.out & 15) == 0) && (e.ldo % 8 == 0);
    constexpr int OC8_G = BN / 16, OC8_T = BN / 8;  // 8-column chunks per row (GeGLU, others)
    static_assert(NT % OC8_T == 0, "fixed output chunk per thread");
    const int oc8 = geglu ? OC8_G : OC8_T;
    const int c8 = tid % oc8;
    float bv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) bv[k] = 0.f;
    if (vec8 && !geglu && e.bias) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (n0 + c8 * 8 + k < N) bv[k] = e.bias[n0 + c8 * 8 + k];
    }
    auto slice = [&](auto ic) {
      const int i = ic;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          sm.c[(wm * 16 + (lane >> 4) * 4 + r) * CLD + wn * WN + j * 16 + (lane & 15)] = acc[i][j][r];
      __syncthreads();
      if (vec8) {
        const int chunks = WGM * 16 * oc8;
        for (int q = tid; q < chunks; q += NT) {
          const int row = q / oc8;
          const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
          if (m >= M) continue;
          const float* cr = sm.c + row * CLD;
          float o[8];
          int col0, total;
          if (geglu) {
            // output column 16 g + j is gate column 32 g + j and up column
            // 32 g + 16 + j of the tile
            const int j0 = c8 * 8, g0 = 32 * (j0 >> 4) + (j0 & 15);
            const float4 ga = *(const float4*)(cr + g0), gb = *(const float4*)(cr + g0 + 4);
            const float4 ua = *(const float4*)(cr + g0 + 16), ub = *(const float4*)(cr + g0 + 20);
            o[0] = gelu_tanh(ga.x) * ua.x;
            o[1] = gelu_tanh(ga.y) * ua.y;
            o[2] = gelu_tanh(ga.z) * ua.z;
            o[3] = gelu_tanh(ga.w) * ua.w;
            o[4] = gelu_tanh(gb.x) * ub.x;
            o[5] = gelu_tanh(gb.y) * ub.y;
            o[6] = gelu_tanh(gb.z) * ub.z;
            o[7] = gelu_tanh(gb.w) * ub.w;
            col0 = n0 / 2 + j0;
            total = N / 2;
          } else {
            const int c0 = c8 * 8;
            const float4 va = *(const float4*)(cr + c0), vb = *(const float4*)(cr + c0 + 4);
            o[0] = va.x + bv[0];
            o[1] = va.y + bv[1];
            o[2] = va.z + bv[2];
            o[3] = va.w + bv[3];
            o[4] = vb.x + bv[4];
            o[5] = vb.y + bv[5];
            o[6] = vb.z + bv[6];
            o[7] = vb.w + bv[7];
            if (ek == EPI_GELU) {
#pragma unroll
              for (int k = 0; k < 8; ++k) o[k] = gelu_tanh(o[k]);
            } else if (ek == EPI_SWISH) {
#pragma unroll
              for (int k = 0; k < 8; ++k) o[k] = swishf(o[k]);
            }
            col0 = n0 + c0;
            total = N;
          }
          T* dst = (T*)e.out + (size_t)m * e.ldo + col0;
          if (col0 + 8 <= total) {
            if constexpr (sizeof(T) == 2) {
              uint4 w;
              w.x = f2bf2(o[0], o[1]);
              w.y = f2bf2(o[2], o[3]);
              w.z = f2bf2(o[4], o[5]);
              w.w = f2bf2(o[6], o[7]);
              *(uint4*)dst = w;
            } else {
              *(float4*)dst = make_float4(o[0], o[1], o[2], o[3]);
              *(float4*)(dst + 4) = make_float4(o[4], o[5], o[6], o[7]);
            }
          } else {
#pragma unroll
            for (int k = 0; k < 8; ++k)
              if (col0 + k < total) TT<T>::st(dst + k, o[k]);
          }
        }
      } else if (fast) {
        constexpr int PER = WGM * 16 * (BN / 2) / NT;
        // f(m, v0, v1) for this thread's rows of the slice (same arithmetic
        // as epi_pair)
        auto each = [&](auto f) {
#pragma unroll 2
          for (int k = 0; k < PER; ++k) {
            const int row = (tid + k * NT) / (BN / 2);
            const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
            if (m < M) {
              float v0 = sm.c[row * CLD + colc], v1 = sm.c[row * CLD + colc + 16];
              if (hasb) {
                v0 += ba;
                v1 += bb;
              }
              f(m, v0, v1);
            }
          }
        };
        // rows' operands that the epilogue reads (RoPE tables, Euler state)
        // are loaded for the whole slice before its first store
        // (in groups of at most 4 rows, for registers)
        auto rows2 = [&](auto ld, auto st) {
          constexpr int RC = PER < 4 ? PER : 4;
#pragma nounroll
          for (int k0 = 0; k0 < PER; k0 += RC) {
          float o0[RC], o1[RC];
#pragma unroll
          for (int k = 0; k < RC; ++k) {
            const int row = (tid + (k0 + k) * NT) / (BN / 2);
            const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
            o0[k] = o1[k] = 0.f;
            if (m < M) ld(m, o0[k], o1[k]);
          }
#pragma unroll
          for (int k = 0; k < RC; ++k) {
            const int row = (tid + (k0 + k) * NT) / (BN / 2);
            const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
            if (m < M) {
              float v0 = sm.c[row * CLD + colc], v1 = sm.c[row * CLD + colc + 16];
              if (hasb) {
                v0 += ba;
                v1 += bb;
              }
              st(m, v0, v1, o0[k], o1[k]);
            }
          }
          }
        };
        constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
        T* out = (T*)e.out;
        // QKV-RoPE with four rotated columns per thread: the four output
        // columns ri .. ri + 3 (and their partners + hd / 2) are contiguous in
        // both Q and the K cache layout, so each goes out as one 8-byte (fp32:
        // 16-byte) store; the V columns keep element stores (the cache layout
        // runs along the keys there). Same arithmetic as the pair path below.
        constexpr int VB = 4 * (int)sizeof(T);  // bytes of four elements
        const bool ropev = ROWK && ek == EPI_QKV_ROPE && ((uintptr_t)e.q % VB) == 0 && e.ldq % 4 == 0 &&
                           ((uintptr_t)e.k % VB) == 0 && e.blk_k % 4 == 0 && (e.hd / 2) % 4 == 0 &&
                           ((uintptr_t)e.rope_cos % 16) == 0 && ((uintptr_t)e.rope_sin % 16) == 0;
        if (ropev) {
          constexpr int QPR = BN / 8;        // column quads per row: four in each 32-column group
          constexpr int RPP = NT / QPR;      // rows per pass
          static_assert(NT % QPR == 0 && (WGM * 16) % RPP == 0, "quads per pass");
          const int hd = e.hd, qcols = e.nq * hd, kcols = e.nkv * hd;
          auto st4 = [&](T* dst, const float (&v)[4]) {
            if constexpr (sizeof(T) == 2)
              *(uint2*)dst = make_uint2(f2bf2(v[0], v[1]), f2bf2(v[2], v[3]));
            else
              *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
          };
          for (int r0 = 0; r0 < WGM * 16; r0 += RPP) {
            const int row = r0 + tid / QPR, qd = tid % QPR;
            const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
            const int c0 = (qd >> 2) * 32 + (qd & 3) * 4;  // first-half column of the tile
            const int n = n0 + c0;
            if (m >= M || n >= N) continue;
            const float4 va = *(const float4*)(sm.c + row * CLD + c0);
            const float4 vb = *(const float4*)(sm.c + row * CLD + c0 + 16);
            const float v0[4] = {va.x, va.y, va.z, va.w}, v1[4] = {vb.x, vb.y, vb.z, vb.w};
            const int key = epi_key(e, m);
            if (n < qcols + kcols) {
              const bool isq = n < qcols;
              const int rn = isq ? n : n - qcols;
              const int head = rn / hd, pp = rn - head * hd;
              const int ri = 16 * (pp >> 5) + (pp & 15);
              const size_t t = (size_t)(e.pos0 + key) * (hd / 2) + ri;
              const float4 cs = *(const float4*)(e.rope_cos + t), sn = *(const float4*)(e.rope_sin + t);
              const float c[4] = {cs.x, cs.y, cs.z, cs.w}, sv[4] = {sn.x, sn.y, sn.z, sn.w};
              float a[4], b[4];
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                a[k] = v0[k] * c[k] - v1[k] * sv[k];
                b[k] = v1[k] * c[k] + v0[k] * sv[k];
              }
              if (isq) {
                T* dst = (T*)e.q + (size_t)m * e.ldq + head * hd;
                st4(dst + ri, a);
                st4(dst + ri + hd / 2, b);
              } else {
                T* dst = (T*)e.k + epi_kblk(e, m, e.blk_k);
                st4(dst + kv_kidx(DT, e.kv_nb, hd, head, key, ri), a);
                st4(dst + kv_kidx(DT, e.kv_nb, hd, head, key, ri + hd / 2), b);
              }
            } else {
              const int c = n - qcols - kcols;
              T* dst = (T*)e.v + epi_kblk(e, m, e.blk_v);
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, (c + k) / hd, key, (c + k) % hd), v0[k]);
                TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, (c + 16 + k) / hd, key, (c + 16 + k) % hd), v1[k]);
              }
            }
          }
        } else if (ROWK && (ek == EPI_QKV_ROPE || ek == EPI_QKV_PLAIN)) {
          const int hd = e.hd, qcols = e.nq * hd, kcols = e.nkv * hd;
          if (ek == EPI_QKV_ROPE && na < qcols + kcols) {
            // column pair (na, nb) holds a rotate-half pair (ri, ri + hd / 2)
            const bool isq = na < qcols;
            const int rn = isq ? na : na - qcols;
            const int head = rn / hd, pp = rn - head * hd;
            const int ri = 16 * (pp >> 5) + (pp & 15);
            if (nb < N)
              rows2(
                  [&](int m, float& c, float& sn) {
                    const size_t t = (size_t)(e.pos0 + epi_key(e, m)) * (hd / 2) + ri;
                    c = e.rope_cos[t];
                    sn = e.rope_sin[t];
                  },
                  [&](int m, float v0, float v1, float c, float sn) {
                    const float a = v0 * c - v1 * sn, b = v1 * c + v0 * sn;
                    if (isq) {
                      T* dst = (T*)e.q + (size_t)m * e.ldq + head * hd;
                      TT<T>::st(dst + ri, a);
                      TT<T>::st(dst + ri + hd / 2, b);
                    } else {
                      const int key = epi_key(e, m);
                      T* dst = (T*)e.k + epi_kblk(e, m, e.blk_k);
                      TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, ri), a);
                      TT<T>::st(dst + kv_kidx(DT, e.kv_nb, hd, head, key, ri + hd / 2), b);
                    }
                  });
          } else if (ek == EPI_QKV_ROPE) {
            // V columns
            const int c0 = na - qcols - kcols, c1 = c0 + 16;
            if (nb < N)
              each([&](int m, float v0, float v1) {
                const int key = epi_key(e, m);
                T* dst = (T*)e.v + epi_kblk(e, m, e.blk_v);
                TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, c0 / hd, key, c0 % hd), v0);
                TT<T>::st(dst + kv_vidx(DT, e.kv_nb, hd, c1 / hd, key, c1 % hd), v1);
              });
          } else {
            // EPI_QKV_PLAIN: column c of q, k or v
            auto put = [&](int m, int n, float v) {
              if (n < qcols) {
                TT<T>::st((T*)e.q + (size_t)m * e.ldq + n, v);
              } else if (n < qcols + kcols) {
                const int c = n - qcols;
                TT<T>::st((T*)e.k + epi_kblk(e, m, e.blk_k) +
                              kv_kidx(DT, e.kv_nb, hd, c / hd, epi_key(e, m), c % hd), v);
              } else {
                const int c = n - qcols - kcols;
                TT<T>::st((T*)e.v + epi_kblk(e, m, e.blk_v) +
                              kv_vidx(DT, e.kv_nb, hd, c / hd, epi_key(e, m), c % hd), v);
              }
            };
            each([&](int m, float v0, float v1) {
              if (na < N) put(m, na, v0);
              if (nb < N) put(m, nb, v1);
            });
          }
        } else if (ROWK && ek == EPI_EULER) {
          rows2(
              [&](int m, float& x0, float& x1) {
                const float* xp = e.x + (size_t)m * e.ldx + na;
                if (na < N) x0 = xp[0];
                if (nb < N) x1 = xp[16];
              },
              [&](int m, float v0, float v1, float x0, float x1) {
                float* xp = e.x + (size_t)m * e.ldx + na;
                if (na < N) {
                  const float xn = __builtin_fmaf(e.dt, v0, x0 * e.xs);
                  xp[0] = xn;
                  TT<T>::st((T*)e.xop + out_at<T>(e, m, na, e.ldxop, e.blk_xop), xn);
                }
                if (nb < N) {
                  const float xn = __builtin_fmaf(e.dt, v1, x1 * e.xs);
                  xp[16] = xn;
                  TT<T>::st((T*)e.xop + out_at<T>(e, m, nb, e.ldxop, e.blk_xop), xn);
                }
              });
        } else if (ek == EPI_GEGLU) {
          const int gcol = 16 * (na >> 5) + (na & 15);
          if (nb < N)
            each([&](int m, float v0, float v1) {
              TT<T>::st(out + out_at<T>(e, m, gcol, e.ldo, e.blk_out), gelu_tanh(v0) * v1);
            });
        } else if (ek == EPI_F32) {
          each([&](int m, float v0, float v1) {
            float* o = (float*)e.out + (size_t)m * e.ldo + na;
            if (na < N) o[0] = v0;
            if (nb < N) o[16] = v1;
          });
        } else {
          // EPI_T, EPI_GELU, EPI_SWISH
          each([&](int m, float v0, float v1) {
            if (ek == EPI_GELU) {
              v0 = gelu_tanh(v0);
              v1 = gelu_tanh(v1);
            } else if (ek == EPI_SWISH) {
              v0 = swishf(v0);
              v1 = swishf(v1);
            }
            if (na < N) TT<T>::st(out + out_at<T>(e, m, na, e.ldo, e.blk_out), v0);
            if (nb < N) TT<T>::st(out + out_at<T>(e, m, nb, e.ldo, e.blk_out), v1);
          });
        }
      } else if (direct) {
        constexpr int PAIRS = WGM * 16 * (BN / 2);  // (row, 32-column group, j < 16)
        for (int p = tid; p < PAIRS; p += NT) {
          const int row = p / (BN / 2), q = p % (BN / 2);
          const int col = (q >> 4) * 32 + (q & 15);
          const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15);
          epi_pair<T, KIND>(e, M, N, m, n0 + col, sm.c[row * CLD + col], sm.c[row * CLD + col + 16]);
        }
      } else if (N % 4 == 0 && ((uintptr_t)P & 15) == 0) {
        // raw fp32 partial of split s: [splits][M][N], four columns per
        // 16-byte store
        for (int p = tid; p < WGM * 16 * (BN / 4); p += NT) {
          const int row = p / (BN / 4), col = (p % (BN / 4)) * 4;
          const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15), n = n0 + col;
          if (m < M && n < N) *(float4*)(P + (size_t)m * N + n) = *(const float4*)(sm.c + row * CLD + col);
        }
      } else {
        // raw fp32 partial of split s: [splits][M][N]
        for (int p = tid; p < WGM * 16 * BN; p += NT) {
          const int row = p / BN, col = p % BN;
          const int m = m0 + (row >> 4) * WM + i * 16 + (row & 15), n = n0 + col;
          if (m < M && n < N) P[(size_t)m * N + n] = sm.c[row * CLD + col];
        }
      }
    };
    // a compile-time loop keeps acc indexed by constants
    static_for<0, TM>(slice);
  }
  VLA_WAVE_END(KK_GEMM);
}

// Sum of split-K partials in split order, then the epilogue.
template <typename T>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ part, int splits,
                                                       int M, int N, Epi e) {
  VLA_WAVE_BEGIN(KK_SPLITK);
  const int groups = (N + 31) / 32;
  const long long total = (long long)M * groups * 16;
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int j = (int)(idx & 15);
    const long long t = idx >> 4;
    const int g = (int)(t % groups), m = (int)(t / groups);
    const int n = g * 32 + j;
    float v0 = 0.f, v1 = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float* P = part + (size_t)s * M * N + (size_t)m * N;
      if (n < N) v0 += P[n];
      if (n + 16 < N) v1 += P[n + 16];
    }
    epi_pair<T>(e, M, N, m, n, v0, v1);
  }
  VLA_WAVE_END(KK_SPLITK);
}

// ---------------------------------------------------------------------------
// Skinny GEMM for M <= 64 (the action expert's rows): C[M, N] = A[M, K] W^T
// with W stored in MFMA fragment order (see frag_index): the 16 x SW fragment
// of n-block nb and K-slab ks is 1 KB contiguous, lane l holding W[16 nb +
// l % 16][SW ks + VEC (l / 16) ...], and A in the row-block operand layout
// (afrag_index), so both operands load as contiguous 1 KB chunks (lda is
// unused). A workgroup owns 32 columns (two
// n-blocks, so the paired epilogues stay inside it) and a K-range of
// 4 * SPW slabs; each wave takes SPW consecutive slabs and issues every load
// of its range at once (one memory round trip), then the four waves' partial
// sums are added in wave order through LDS. K-ranges beyond one workgroup
// are split: EPI_PART leaves the split partials to the consumer, other
// epilogues go through the split-K reduce kernel.
// ---------------------------------------------------------------------------

// The last split of a 32-column pair of a folded-norm producer (one frame):
// thread t takes row t / 4 and columns 8 (t % 4) .. + 7 of the pair; the
// pair's split partials are summed in split order (all loads in flight at
// once) and added to the residual x, as the norm kernel adds them; then the
// operand x * g and the row's sum of squares over the pair's columns (eight
// in order per thread, then the row's four threads in order) are written.
template <typename T>
__device__ __forceinline__ void fold_pair(const Epi& e, int np, int M, int N, int splits, int tid,
                                          float (&sPart)[64][4]) {
  constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
  constexpr int MAXS = 8;  // splits (checked on the host)
  const int row = tid >> 2, c0 = np * 32 + (tid & 3) * 8;
  const bool ok = row < M && c0 < N;
  const Rsrc rp = rsrc(e.out, (size_t)splits * M * N * 4);
  f32x4 pa[MAXS], pb[MAXS];
#pragma unroll
  for (int q = 0; q < MAXS; ++q) {
    const uint32_t off = (uint32_t)((((size_t)q * M + row) * N + c0) * 4);
    const bool okq = ok && q < splits;
    pa[q] = bld16_sc1(rp, okq ? off : OOB);
    pb[q] = bld16_sc1(rp, okq ? off + 16 : OOB);
  }
  const Rsrc rx = rsrc(e.x, span(M, e.ldx, N, 4));
  const Rsrc rg = rsrc(e.norm_g, (size_t)N * 4);
  const uint32_t xo = (uint32_t)(((size_t)row * e.ldx + c0) * 4);
  f32x4 xa = bld4f(rx, ok ? xo : OOB), xb = bld4f(rx, ok ? xo + 16 : OOB);
  const f32x4 ga = bld4f(rg, ok ? (uint32_t)(c0 * 4) : OOB), gb = bld4f(rg, ok ? (uint32_t)(c0 * 4 + 16) : OOB);
  f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = sa;
#pragma unroll
  for (int q = 0; q < MAXS; ++q)
    if (q < splits) {
      sa += pa[q];
      sb += pb[q];
    }
  xa += sa;
  xb += sb;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < 4; ++k) ss += xa[k] * xa[k];
#pragma unroll
  for (int k = 0; k < 4; ++k) ss += xb[k] * xb[k];
  if (ok) {
    *(f32x4*)(e.x + (size_t)row * e.ldx + c0) = xa;
    *(f32x4*)(e.x + (size_t)row * e.ldx + c0 + 4) = xb;
    const f32x4 ya = xa * ga, yb = xb * gb;
    if constexpr (sizeof(T) == 2) {
      *(uint4*)((T*)e.norm_out + afrag_index(DT, row, c0)) =
          make_uint4(f2bf2(ya[0], ya[1]), f2bf2(ya[2], ya[3]), f2bf2(yb[0], yb[1]), f2bf2(yb[2], yb[3]));
    } else {
      *(f32x4*)((T*)e.norm_out + afrag_index(DT, row, c0)) = ya;
      *(f32x4*)((T*)e.norm_out + afrag_index(DT, row, c0 + 4)) = yb;
    }
  }
  sPart[row][tid & 3] = ss;
  __syncthreads();
  if ((tid & 3) == 0 && row < M)
    e.rowss[(size_t)np * M + row] = ((sPart[row][0] + sPart[row][1]) + sPart[row][2]) + sPart[row][3];
  __syncthreads();  // sPart is free again
}

// Frames (a batched action phase): `frames` row blocks of M rows, block f of
// A at A + f a_blk elements. Every (column pair, K-range) tile is computed
// once per frame by its own workgroup, exactly as in a one-frame call; the
// frames of a tile are consecutive tile indices, and with the XCD-aware
// order below they run on one XCD at the same time, so the weights come
// from HBM once and from that XCD's L2 for the other frame.
// One instantiation per epilogue kind (KIND): the action loop launches these
// kernels back to back, and each carries only its own epilogue's code, which
// keeps the code the loop runs small enough to stay in the instruction cache.
template <typename T, int SPW, int KIND>
__global__ __launch_bounds__(256) void k_skinny(const T* __restrict__ A, size_t a_blk, int frames,
                                                const T* __restrict__ Wf, int KS, int ks0, int M,
                                                int N, int K, int splits, Epi e,
                                                float* __restrict__ part) {
  VLA_WAVE_BEGIN(KK_SKINNY);
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SW = 4 * VEC;
  __shared__ float red[4][8][4][64];  // [wave][n-block * 4 + m-tile][r][lane]
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int npairs = (N + 31) / 32;
  const int nslab = (K + SW - 1) / SW;
  const int total = npairs * splits * frames;
  const int Mt = M * frames;  // rows of all frames
  const T dummy = T();
  const Rsrc rw = rsrc(Wf, (size_t)npairs * 2 * KS * 64 * VEC * sizeof(T));
  // row-block operand layout, one block per frame
  const Rsrc ra = rsrc(A, ((size_t)(frames - 1) * a_blk + (size_t)nslab * 4 * 64 * VEC) * sizeof(T));
  const int G = gridDim.x;
  const int first = frames > 1 && G % 8 == 0 ? (int)(blockIdx.x % 8) * (G / 8) + (int)(blockIdx.x / 8)
                                             : (int)blockIdx.x;
  // Folded RMSNorm (see Epi::rowss). Consumer: thread t holds the partial
  // sums of squares of row t / 4 for the pairs congruent to t % 4 (mod 4),
  // requested before the first tile's loads (waiting for those covers them)
  // and turned into the rows' scales at the first epilogue.
  __shared__ float sPart[64][4];
  __shared__ float sInv[64];
  __shared__ int sLast;
  constexpr int SSQ = 16;  // pairs per thread: at most 64 pairs
  const bool rowscale = KIND != EPI_PART && e.rowss != nullptr;
  const int srow = tid >> 2, squ = tid & 3;
  float ssq[SSQ];
  if (rowscale) {
    const Rsrc rs = rsrc(e.rowss, (size_t)e.rowss_n * M * 4);
#pragma unroll
    for (int k = 0; k < SSQ; ++k) {
      const int p = squ + 4 * k;
      ssq[k] = bld1(rs, p < e.rowss_n && srow < M ? (uint32_t)(((size_t)p * M + srow) * 4) : OOB);
    }
  }
  bool inv_ready = false;
  for (int w = first; w < total; w += G) {
    const int f = w % frames, wt = w / frames;
    const int s = wt % splits, np = wt / splits;
    const int sb = (s * 4 + wave) * SPW;
    const uint32_t aoff = (uint32_t)((size_t)f * a_blk * sizeof(T));  // frame f's block
    uint4 bf[SPW][2], af[SPW][4];
#pragma unroll
    for (int q = 0; q < SPW; ++q) {
      const int ks = sb + q;
      const bool ok = ks < nslab;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        bf[q][nb] = bld16(rw, ok ? (uint32_t)((((size_t)(2 * np + nb) * KS + ks0 + ks) * 64 + lane) * VEC * sizeof(T))
                                 : OOB);
      const int k = ks * SW + (lane >> 4) * VEC;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = mt * 16 + (lane & 15);
        const bool oka = ok && row < M && k < K;
        af[q][mt] = bld16s(ra, oka ? (uint32_t)((((size_t)ks * 4 + mt) * 64 + lane) * VEC * sizeof(T)) : OOB, aoff);
      }
    }
    f32x4 acc[2][4];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) acc[nb][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < SPW; ++q)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[nb][mt] = mfma_step(af[q][mt], bf[q][nb], acc[nb][mt], dummy);

    __syncthreads();  // red is free (previous tile's epilogue done)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][nb * 4 + mt][r][lane] = acc[nb][mt][r];
    __syncthreads();
    // wave w finishes m-tile w: sum the four waves in order, then the epilogue
    const int mt = wave;
    const int n = np * 32 + (lane & 15);
    int mg[4], nn[4];
    float v0[4], v1[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      v0[r] = ((red[0][mt][r][lane] + red[1][mt][r][lane]) + red[2][mt][r][lane]) + red[3][mt][r][lane];
      v1[r] = ((red[0][4 + mt][r][lane] + red[1][4 + mt][r][lane]) + red[2][4 + mt][r][lane]) +
              red[3][4 + mt][r][lane];
      const int m = mt * 16 + (lane >> 4) * 4 + r;
      mg[r] = m < M ? f * M + m : Mt;  // row over all frames (Mt: skipped)
      nn[r] = n;
    }
    if (rowscale) {
      if (!inv_ready) {
        float t = 0.f;
#pragma unroll
        for (int k = 0; k < SSQ; ++k) t += ssq[k];  // pairs in increasing order (absent ones read 0)
        sPart[srow][squ] = t;
        __syncthreads();
        if (squ == 0)
          sInv[srow] = 1.f / sqrtf((((sPart[srow][0] + sPart[srow][1]) + sPart[srow][2]) + sPart[srow][3]) /
                                       e.rowss_d + 1e-6f);
        __syncthreads();
        inv_ready = true;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = mt * 16 + (lane >> 4) * 4 + r;
        const float sc = sInv[m];
        v0[r] *= sc;
        v1[r] *= sc;
      }
    }
    if (KIND != EPI_PART && splits == 1) {
      epi_pairs<T, 4, KIND>(e, Mt, N, mg, nn, v0, v1);
    } else {
      const bool fold = KIND == EPI_PART && e.norm_g != nullptr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (mg[r] >= Mt) continue;
        float* P = (KIND == EPI_PART ? (float*)e.out : part) + (size_t)s * Mt * N + (size_t)mg[r] * N;
        if (fold) {
          // write-through: the pair's last split, on any XCD, reads them
          if (n < N) __hip_atomic_store((uint32_t*)P + n, __float_as_uint(v0[r]), __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT);
          if (n + 16 < N) __hip_atomic_store((uint32_t*)P + n + 16, __float_as_uint(v1[r]), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        } else {
          if (n < N) P[n] = v0[r];
          if (n + 16 < N) P[n + 16] = v1[r];
        }
      }
      if constexpr (KIND == EPI_PART) {
        if (fold) {
          // Every thread's partial stores have completed (vmcnt counts
          // stores here) before thread 0 counts this split in; the split
          // that counts last finishes the pair. No split waits for another.
          __builtin_amdgcn_s_waitcnt(VMCNT0);
          __syncthreads();
          if (tid == 0) {
            const unsigned old = __hip_atomic_fetch_add(e.cnt + np, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            sLast = old == (unsigned)(splits - 1);
            // back to zero for the next launch (and graph replay)
            if (sLast) __hip_atomic_store(e.cnt + np, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          }
          __syncthreads();
          if (sLast) fold_pair<T>(e, np, M, N, splits, tid, sPart);
        }
      }
    }
  }
  VLA_WAVE_END(KK_SKINNY);
}

// Row-major copy of a fragment-ordered weight: one thread per 16-byte piece
// (VEC consecutive k of one row n, which the fragment order keeps together).
template <typename T>
__global__ __launch_bounds__(256) void k_unfrag(const T* __restrict__ Wf, int N, int K, int KS,
                                                T* __restrict__ out) {
  constexpr int VEC = 16 / sizeof(T), SW = 4 * VEC;
  const int kv = K / VEC;
  const long long total = (long long)N * kv;
  for (long long i = blockIdx.x * (long long)blockDim.x + threadIdx.x; i < total;
       i += (long long)gridDim.x * blockDim.x) {
    const int n = (int)(i / kv), k = (int)(i % kv) * VEC;
    const size_t frag = (size_t)(n / 16) * KS + k / SW;
    const int lane = n % 16 + 16 * ((k % SW) / VEC);
    *(uint4*)(out + (size_t)n * K + k) = *(const uint4*)(Wf + (frag * 64 + lane) * VEC);
  }
}

// Copy in 16-byte pieces when both pointers and the size allow it, else in
// bytes.
__global__ __launch_bounds__(256) void k_copy16(uint4* __restrict__ dst, const uint4* __restrict__ src, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}
__global__ __launch_bounds__(256) void k_copy1(unsigned char* __restrict__ dst, const unsigned char* __restrict__ src,
                                               size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  if (!dst || !src) return hipErrorInvalidValue;
  if (((uintptr_t)dst | (uintptr_t)src | bytes) % 16 == 0) {
    const size_t n = bytes / 16;
    const int grid = (int)std::min<size_t>((n + 255) / 256, 1024);
    k_copy16<<<grid, 256, 0, st>>>((uint4*)dst, (const uint4*)src, n);
  } else {
    const int grid = (int)std::min<size_t>((bytes + 255) / 256, 1024);
    k_copy1<<<grid, 256, 0, st>>>((unsigned char*)dst, (const unsigned char*)src, bytes);
  }
  return hipGetLastError();
}

hipError_t launch_unfrag(int dtype, const void* frag, int N, int K, int KS, void* out, hipStream_t st) {
  const int vec = dtype == DT_BF16 ? 8 : 4;
  if (N <= 0 || K <= 0 || K % vec || KS * frag_slab(dtype) < K) return hipErrorInvalidValue;
  const long long total = (long long)N * (K / vec);
  const int grid = (int)std::min<long long>((total + 255) / 256, 8192);
  if (dtype == DT_BF16)
    k_unfrag<uint16_t><<<grid, 256, 0, st>>>((const uint16_t*)frag, N, K, KS, (uint16_t*)out);
  else
    k_unfrag<float><<<grid, 256, 0, st>>>((const float*)frag, N, K, KS, (float*)out);
  return hipGetLastError();
}

size_t frag_index(int n, int k, int KS, int dtype) {
  const int vec = dtype == DT_BF16 ? 8 : 4, sw = 4 * vec;
  const size_t frag = (size_t)(n / 16) * KS + k / sw;
  const int lane = n % 16 + 16 * ((k % sw) / vec);
  return (frag * 64 + lane) * vec + k % vec;
}

int frag_slab(int dtype) { return dtype == DT_BF16 ? 32 : 16; }

static int skinny_spw(const GemmDesc& g) { return g.epi.kind == EPI_PART ? 4 : 8; }

int skinny_splits(const GemmDesc& g) {
  const int sw = frag_slab(g.dtype);
  const int per_wg = 4 * skinny_spw(g) * sw;
  return std::max(1, (g.K + per_wg - 1) / per_wg);
}

template <typename T, int SPW, int KIND>
static hipError_t run_skinny_t(const GemmDesc& g, int splits, const Scratch& s,
                               const LaunchCaps& caps, hipStream_t st) {
  int grid = ((g.N + 31) / 32) * splits * g.frames;
  if (caps.max_wgs > 0) grid = std::min(grid, caps.max_wgs);
  hipExtLaunchKernelGGL((k_skinny<T, SPW, KIND>), dim3(grid), dim3(256), 0, st, caps.ev_start,
                        caps.ev_stop, 0, (const T*)g.A, g.a_blk, g.frames, (const T*)g.W, g.frag_ks,
                        g.frag_ks0, g.M, g.N, g.K, splits, g.epi, s.ptr);
  if (splits > 1 && g.epi.kind != EPI_PART) {
    const int Mt = g.M * g.frames;
    const long long total = (long long)Mt * ((g.N + 31) / 32) * 16;
    int rgrid = (int)std::min<long long>((total + 255) / 256, 4096);
    if (caps.max_wgs > 0) rgrid = std::min(rgrid, caps.max_wgs);
    k_splitk_reduce<T><<<rgrid, 256, 0, st>>>(s.ptr, splits, Mt, g.N, g.epi);
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t run_skinny_kind(const GemmDesc& g, int splits, const Scratch& s, const LaunchCaps& caps,
                                  hipStream_t st) {
  switch (g.epi.kind) {
    case EPI_F32: return run_skinny_t<T, 8, EPI_F32>(g, splits, s, caps, st);
    case EPI_T: return run_skinny_t<T, 8, EPI_T>(g, splits, s, caps, st);
    case EPI_RESID: return run_skinny_t<T, 8, EPI_RESID>(g, splits, s, caps, st);
    case EPI_GELU: return run_skinny_t<T, 8, EPI_GELU>(g, splits, s, caps, st);
    case EPI_SWISH: return run_skinny_t<T, 8, EPI_SWISH>(g, splits, s, caps, st);
    case EPI_GEGLU: return run_skinny_t<T, 8, EPI_GEGLU>(g, splits, s, caps, st);
    case EPI_QKV_ROPE: return run_skinny_t<T, 8, EPI_QKV_ROPE>(g, splits, s, caps, st);
    case EPI_QKV_PLAIN: return run_skinny_t<T, 8, EPI_QKV_PLAIN>(g, splits, s, caps, st);
    case EPI_EULER: return run_skinny_t<T, 8, EPI_EULER>(g, splits, s, caps, st);
    case EPI_PART: return run_skinny_t<T, 4, EPI_PART>(g, splits, s, caps, st);
    default: return hipErrorInvalidValue;
  }
}

static hipError_t launch_skinny(const GemmDesc& g, const Scratch& s, const LaunchCaps& caps,
                                hipStream_t st) {
  if (g.M > 64 || g.frames < 1 || g.frames > MAX_FRAMES ||
      (g.frames > 1 && (g.epi.blk_rows != g.M || g.a_blk < afrag_elems(g.dtype, g.K))))
    return hipErrorInvalidValue;
  const int splits = skinny_splits(g);
  const size_t need = (size_t)splits * g.M * g.frames * g.N;
  const Epi& e = g.epi;
  // folded RMSNorm (Epi::rowss): one frame; a producer's partials in at most
  // 8 splits, whole 8-column groups, its operand output in the row-block
  // layout; a consumer's product unsplit (the scale precedes the epilogue)
  if (e.kind == EPI_PART && e.norm_g &&
      (g.frames != 1 || splits > 8 || g.N % 8 || (g.N + 31) / 32 > 64 || !e.x || e.ldx < g.N || !e.norm_out ||
       !e.rowss || !e.cnt || !e.afrag))
    return hipErrorInvalidValue;
  if (e.kind != EPI_PART && e.rowss &&
      (g.frames != 1 || splits != 1 || e.rowss_n < 1 || e.rowss_n > 64 || e.rowss_d < 1))
    return hipErrorInvalidValue;
  if (g.epi.kind == EPI_PART) {
    if (!g.epi.out || need > (size_t)g.epi.ldo) return hipErrorInvalidValue;
  } else if (splits > 1 && need > s.floats) {
    return hipErrorInvalidValue;
  }
  if (g.dtype == DT_BF16) return run_skinny_kind<uint16_t>(g, splits, s, caps, st);
  return run_skinny_kind<float>(g, splits, s, caps, st);
}

struct TileCfg {
  int bm, bn, bk;
};
// bf16 configurations, then fp32 ones. Wide GEMMs (enough 128 x 128 tiles to
// cover every CU) take the large tile; everything else takes 64 x 64 tiles,
// which keep more loads in flight per CU for these M ~ 256..320 shapes.
static const TileCfg kBf16Cfg[] = {{128, 128, 64}, {64, 64, 64}, {32, 64, 64}, {256, 256, 64}};
static const TileCfg kF32Cfg[] = {{64, 64, 32}, {32, 64, 32}};

GemmPlan plan_gemm(const GemmDesc& g) {
  GemmPlan p{};
  if (g.frag_ks > 0) {  // fragment-ordered weights: skinny kernel
    p.cfg = -1;
    p.splits = skinny_splits(g);
    p.tiles = ((g.N + 31) / 32) * p.splits * g.frames;
    p.scratch_floats = (p.splits > 1 || g.epi.kind == EPI_PART) ? (size_t)p.splits * g.M * g.frames * g.N : 0;
    return p;
  }
  const TileCfg* cfgs = g.dtype == DT_BF16 ? kBf16Cfg : kF32Cfg;
  // The 256 x 256 tile does about twice the work per CU-cycle of the
  // 128 x 128 tile (one workgroup per CU at ~3,600 cycles per K-step against
  // two at ~3,900), so where it leaves CUs idle it can still win: with the
  // epilogues that take its short paths (GeGLU, store, GELU, swish) it is
  // also chosen when its rounds of tiles take fewer cycles than the 128
  // tile's, counting ~18K cycles of epilogue per 256 tile. The tile does not
  // change any sum (same BK, same splits), only which workgroup computes it.
  const int kb64 = (g.K + 63) / 64;
  const bool cheap_epi = g.epi.kind == EPI_GEGLU || g.epi.kind == EPI_T || g.epi.kind == EPI_GELU ||
                         g.epi.kind == EPI_SWISH;
  // Split-K partials of `splits` K-ranges of kc 64-wide blocks each also go
  // to the 256 tile when its workgroups make exactly one round on the chip
  // (at least 7/8 of it) and each split is long enough (kc >= 10) to carry
  // the partial epilogue; a second, partly empty round of 256 tiles loses to
  // the 128 tile, a single full one wins (measured alone, weights from HBM:
  // 2440 x 2048 x 2048 in 3 splits of kc 11, 35 us against 51 us on the
  // 128 tile; 2048 x 1152 x 4304 in 6 splits of kc 12, 40 us against 51 us
  // on the 64 tile; with kc 3 the 256 tile loses).
  auto part256 = [&](int t256, int splits) {
    const int kc = (kb64 + splits - 1) / splits;
    return g.epi.kind == EPI_PART && splits > 0 && kc >= 10 && t256 * splits <= NUM_CU_PLAN &&
           t256 * splits >= NUM_CU_PLAN * 7 / 8;
  };
  auto choose = [&](int M, int splits) {
    if (g.dtype == DT_BF16) {
      const int t128 = ((M + 127) / 128) * ((g.N + 127) / 128);
      const int t256 = ((M + 255) / 256) * ((g.N + 255) / 256);
      if (M >= 1024 && t256 >= NUM_CU_PLAN) return 3;
      if (M >= 1024 && part256(t256, splits)) return 3;
      if (M >= 1024 && cheap_epi) {
        const long long c256 = (long long)((t256 + NUM_CU_PLAN - 1) / NUM_CU_PLAN) * (kb64 * 3600LL + 18000);
        const long long c128 = (long long)((t128 + 2 * NUM_CU_PLAN - 1) / (2 * NUM_CU_PLAN)) * (kb64 * 3900LL);
        if (c256 < c128) return 3;
      }
      if (M >= 256 && t128 >= NUM_CU_PLAN) return 0;
      return M > 32 ? 1 : 2;
    }
    return M > 32 ? 0 : 1;
  };
  // The split factor comes from the rows of one frame (plan_m), the tile
  // from all M rows; every configuration of a dtype has the same BK, so the
  // K range of each split (and every sum) is the same as in a one-frame call.
  const int Mp = g.plan_m > 0 ? g.plan_m : g.M;  // may exceed M (a fixed reference row count)
  // (the split count is planned first, from the tile of Mp rows chosen as
  // if unsplit; every tile of a dtype has the same BK)
  const TileCfg tp = cfgs[choose(Mp, 0)];
  const int tiles = ((Mp + tp.bm - 1) / tp.bm) * ((g.N + tp.bn - 1) / tp.bn);
  const int kblocks = (g.K + tp.bk - 1) / tp.bk;
  // Split K where it is free: partial sums (EPI_PART) are added by their
  // consumer, so aim for at most two workgroups per CU with at least four
  // K-blocks each (rounded down: 408 x 1024 x 4096 on the 64 tile, measured
  // alone, 12.6 us in 4 splits against 14.4 us in 5). Other epilogues need a separate reduction pass, so only very
  // small tile counts are split.
  int splits = 1;
  if (g.epi.kind == EPI_PART && tiles < 2 * NUM_CU_PLAN)
    splits = std::min(std::max(1, 2 * NUM_CU_PLAN / tiles), std::max(1, kblocks / 4));
  else if (tiles < 32 && kblocks >= 16)
    splits = std::min(NUM_CU_PLAN / tiles, kblocks / 4);
  splits = std::max(splits, 1);
  // Fewer splits where that lets the largest batched launch of the plan
  // (plan_batch x Mp rows, a prefill batch) run on the 256 tile in one round
  // (part256): the most splits below the planned count that do; the count
  // stays the same for every batch size.
  if (g.dtype == DT_BF16 && g.plan_batch > 1 && splits > 1) {
    const int Mb = g.plan_batch * Mp;
    const int t256b = ((Mb + 255) / 256) * ((g.N + 255) / 256);
    if (Mb >= 1024 && !part256(t256b, splits))
      for (int s2 = splits - 1; s2 >= 1; --s2)
        if (part256(t256b, s2)) {
          splits = s2;
          break;
        }
    // One split where that batched launch fills the chip twice over unsplit
    // and K is short (at most 32 K-tiles): splitting then only adds partial
    // traffic (2048 x 1152 x 1152 on the 64 tile, measured alone: 16.8 us
    // unsplit against 19.9 us in 4 splits, and the consumer reads a quarter)
    if (!part256(t256b, splits) && kblocks <= 32) {
      const TileCfg tb = cfgs[choose(Mb, 1)];
      if (((Mb + tb.bm - 1) / tb.bm) * ((g.N + tb.bn - 1) / tb.bn) >= 2 * NUM_CU_PLAN) splits = 1;
    }
  }
  const int kchunk_blocks = (kblocks + splits - 1) / splits;
  splits = (kblocks + kchunk_blocks - 1) / kchunk_blocks;
  const int c = choose(g.M, splits);
  const TileCfg t = cfgs[c];
  p.cfg = c;
  p.splits = splits;
  p.tiles = ((g.M + t.bm - 1) / t.bm) * ((g.N + t.bn - 1) / t.bn) * splits;
  p.scratch_floats = (splits > 1 || g.epi.kind == EPI_PART) ? (size_t)splits * g.M * g.N : 0;
  return p;
}

void plan_tile(const GemmDesc& g, const GemmPlan& p, int* bm, int* bn) {
  if (p.cfg < 0) {
    *bm = 0;
    *bn = 32;
    return;
  }
  const TileCfg t = (g.dtype == DT_BF16 ? kBf16Cfg : kF32Cfg)[p.cfg];
  *bm = t.bm;
  *bn = t.bn;
}

template <typename T, int BM, int BN, int BK, int WGM = 2, int WGN = 2, int PD = 1, int PAD = VLA_GEMM_LDS_PAD,
          bool DL = false, int KIND = -1>
static hipError_t run_gemm_t(const GemmDesc& g, const GemmPlan& p, const Scratch& s,
                             const LaunchCaps& caps, hipStream_t st) {
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const int kblocks = (g.K + BK - 1) / BK;
  const int kchunk = ((kblocks + p.splits - 1) / p.splits) * BK;
  int grid = p.tiles;
  if (caps.max_wgs > 0) grid = std::min(grid, caps.max_wgs);
  // row-tile bands sized so a band's A K-range takes about half of an XCD's
  // 4 MB L2
  const size_t band_bytes = (size_t)BM * kchunk * sizeof(T);
  const int group_m = std::max(1, std::min(tiles_m, (int)((2u << 20) / std::max<size_t>(band_bytes, 1))));
  hipExtLaunchKernelGGL((k_gemm<T, BM, BN, BK, WGM, WGN, PD, PAD, DL, KIND>), dim3(grid), dim3(64 * WGM * WGN), 0, st,
                        caps.ev_start,
                        caps.ev_stop, 0, (const T*)g.A, g.lda, (const T*)g.W, g.ldw, g.M, g.N,
                        g.K, kchunk, p.splits, tiles_m, tiles_n, group_m, g.epi, s.ptr);
  if (p.splits > 1 && g.epi.kind != EPI_PART) {
    const long long total = (long long)g.M * ((g.N + 31) / 32) * 16;
    int rgrid = (int)std::min<long long>((total + 255) / 256, 4096);
    if (caps.max_wgs > 0) rgrid = std::min(rgrid, caps.max_wgs);
    k_splitk_reduce<T><<<rgrid, 256, 0, st>>>(s.ptr, p.splits, g.M, g.N, g.epi);
  }
  return hipGetLastError();
}

// the 4-wave tiles: the decoder layers' epilogues (QKV-RoPE, GeGLU, split-K
// partials) get their own instantiations, the rest share the run-time one
template <typename T, int BM, int BN, int BK, int PD, int PAD = VLA_GEMM_LDS_PAD, bool DL = false>
static hipError_t run_gemm_kind(const GemmDesc& g, const GemmPlan& p, const Scratch& s, const LaunchCaps& caps,
                                hipStream_t st) {
  switch (g.epi.kind) {
    case EPI_QKV_ROPE: return run_gemm_t<T, BM, BN, BK, 2, 2, PD, PAD, DL, EPI_QKV_ROPE>(g, p, s, caps, st);
    case EPI_GEGLU: return run_gemm_t<T, BM, BN, BK, 2, 2, PD, PAD, DL, EPI_GEGLU>(g, p, s, caps, st);
    case EPI_PART: return run_gemm_t<T, BM, BN, BK, 2, 2, PD, PAD, DL, EPI_PART>(g, p, s, caps, st);
    default: return run_gemm_t<T, BM, BN, BK, 2, 2, PD, PAD, DL>(g, p, s, caps, st);
  }
}

hipError_t launch_gemm(const GemmDesc& g, const Scratch& s, const LaunchCaps& caps,
                       hipStream_t st) {
  if (g.frag_ks > 0) return launch_skinny(g, s, caps, st);
  const GemmPlan p = plan_gemm(g);
  if (g.epi.kind == EPI_PART) {
    if (!g.epi.out || (size_t)p.splits * g.M * g.N > (size_t)g.epi.ldo) return hipErrorInvalidValue;
  } else if (p.scratch_floats > s.floats) {
    return hipErrorInvalidValue;
  }
  if (g.dtype == DT_BF16) {
    switch (p.cfg) {
      case 0: return run_gemm_kind<uint16_t, 128, 128, 64, 3>(g, p, s, caps, st);
      case 1: return run_gemm_kind<uint16_t, 64, 64, 64, 2>(g, p, s, caps, st);
      case 3: return run_gemm_t<uint16_t, 256, 256, 64, 2, 4, 1, 0, true>(g, p, s, caps, st);
      default: return run_gemm_kind<uint16_t, 32, 64, 64, 2>(g, p, s, caps, st);
    }
  }
  switch (p.cfg) {
    case 0: return run_gemm_t<float, 64, 64, 32, 2, 2, 2>(g, p, s, caps, st);
    default: return run_gemm_t<float, 32, 64, 32, 2, 2, 2>(g, p, s, caps, st);
  }
}

// ---------------------------------------------------------------------------
// Attention: unmasked softmax(q k^T / sqrt(hd)) v with grouped KV heads and
// keys from two segments [k0; k1]. The rows of one KV head's query heads are
// packed (row r <-> query r / group, head r % group), 64 packed rows per
// workgroup, 16 per wave. Keys stream in blocks of 32 through LDS (V stored
// transposed); scores and the online softmax are fp32. P V runs on MFMA: in
// bf16 with P split into a bf16 high part and a bf16 remainder (two MFMAs,
// so P keeps ~16 significant bits); in fp32 directly. Long key ranges are
// split across workgroups and merged in split order by k_attn_combine.
// ---------------------------------------------------------------------------

constexpr int ATT_BQ = 64, ATT_BKV = 32;

struct AttnArgs {
  const void* q;
  const void* k0;
  const void* v0;
  const void* k1;
  const void* v1;
  void* out;
  float* po;  // partial outputs [work][splits][64][HDP]
  float* pm;  // partial row max (log2 domain) [work][splits][64]
  float* pl;  // partial row sums
  int ldq, ldkv, ldo, Sq, nq, nkv, hd, S0, S1, segs, splits, qblocks;
  long long seg_q, seg_kv, seg_o;
  float scale_log2;
};

template <typename T, int HDP>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  VLA_WAVE_BEGIN(KK_ATTN);
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SW = 4 * VEC;
  constexpr int KS = HDP + VEC;          // sK row stride
  constexpr int VS = ATT_BKV + VEC;      // sVt row stride
  constexpr int PS = ATT_BKV + 4;        // sP row stride (fp32)
  constexpr int NQF = HDP / SW;          // Q fragments per lane
  constexpr int NOT = HDP / 16;          // output tiles per wave
  __shared__ __attribute__((aligned(16))) T sK[ATT_BKV * KS];
  __shared__ __attribute__((aligned(16))) T sVt[HDP * VS];
  __shared__ __attribute__((aligned(16))) float sP[4 * 16 * PS];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int group = a.nq / a.nkv;
  const int R = a.Sq * group;
  const int Skv = a.S0 + a.S1;
  const int nblk = (Skv + ATT_BKV - 1) / ATT_BKV;
  const int bps = (nblk + a.splits - 1) / a.splits;
  const int total = a.qblocks * a.nkv * a.segs * a.splits;
  const T dummy = T();

  for (int w = blockIdx.x; w < total; w += gridDim.x) {
    const int sp = w % a.splits;
    const int work = w / a.splits;
    int t = work;
    const int qb = t % a.qblocks;
    t /= a.qblocks;
    const int j = t % a.nkv;
    const int seg = t / a.nkv;

    const T* Q = (const T*)a.q + seg * a.seg_q;
    const T* K0 = (const T*)a.k0 + seg * a.seg_kv;
    const T* V0 = (const T*)a.v0 + seg * a.seg_kv;
    const T* K1 = a.k1 ? (const T*)a.k1 + seg * a.seg_kv : K0;
    const T* V1 = a.v1 ? (const T*)a.v1 + seg * a.seg_kv : V0;
    const Rsrc rq = rsrc(Q, span(a.Sq, a.ldq, a.nq * a.hd, sizeof(T)));
    const Rsrc rk0 = rsrc(K0, span(a.S0, a.ldkv, a.nkv * a.hd, sizeof(T)));
    const Rsrc rv0 = rsrc(V0, span(a.S0, a.ldkv, a.nkv * a.hd, sizeof(T)));
    const Rsrc rk1 = rsrc(K1, span(a.S1, a.ldkv, a.nkv * a.hd, sizeof(T)));
    const Rsrc rv1 = rsrc(V1, span(a.S1, a.ldkv, a.nkv * a.hd, sizeof(T)));

    // Q fragments of this lane's packed row (A-operand layout).
    uint4 qf[NQF];
    {
      const int r = qb * ATT_BQ + wave * 16 + (lane & 15);
      const int sq = r / group, h = j * group + r % group;
#pragma unroll
      for (int ks = 0; ks < NQF; ++ks) {
        const int d = ks * SW + (lane >> 4) * VEC;
        const bool ok = r < R && d < a.hd;
        qf[ks] = bld16(rq, ok ? (uint32_t)(((size_t)sq * a.ldq + h * a.hd + d) * sizeof(T)) : OOB);
      }
    }

    float mrow[4], lrow[4];
    f32x4 o[NOT];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      mrow[r] = -INFINITY;
      lrow[r] = 0.f;
    }
#pragma unroll
    for (int d = 0; d < NOT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int b0 = sp * bps, b1 = min(nblk, b0 + bps);
    for (int b = b0; b < b1; ++b) {
      __syncthreads();
      constexpr int NV = ATT_BKV * (HDP / VEC);
      // a block inside segment 0 reads one buffer; a block that reaches into
      // segment 1 reads both with the other one's offset out of range (zero)
      // and merges them, so the buffer choice never depends on the lane
      const bool only0 = (b + 1) * ATT_BKV <= a.S0;
      for (int c = tid; c < NV; c += 256) {
        const int kk = c / (HDP / VEC), d = (c % (HDP / VEC)) * VEC;
        const int key = b * ATT_BKV + kk;
        const bool ok = key < Skv && d < a.hd;
        const bool s0 = key < a.S0;
        const uint32_t off = ok ? (uint32_t)(((size_t)(s0 ? key : key - a.S0) * a.ldkv + j * a.hd + d) *
                                             sizeof(T))
                                : OOB;
        uint4 kv, vv;
        if (only0) {
          kv = bld16(rk0, off);
          vv = bld16(rv0, off);
        } else {
          const uint32_t o0 = s0 ? off : OOB, o1 = s0 ? OOB : off;
          const uint4 ka = bld16(rk0, o0), kb = bld16(rk1, o1);
          const uint4 va = bld16(rv0, o0), vb = bld16(rv1, o1);
          kv = make_uint4(ka.x | kb.x, ka.y | kb.y, ka.z | kb.z, ka.w | kb.w);
          vv = make_uint4(va.x | vb.x, va.y | vb.y, va.z | vb.z, va.w | vb.w);
        }
        *(uint4*)(sK + kk * KS + d) = kv;
        const T* ve = (const T*)&vv;
#pragma unroll
        for (int q = 0; q < VEC; ++q) sVt[(d + q) * VS + kk] = ve[q];
      }
      __syncthreads();

      // scores for 16 rows x 32 keys
      f32x4 sacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int ks = 0; ks < NQF; ++ks) {
          const uint4 kf = *(const uint4*)(sK + (nt * 16 + (lane & 15)) * KS + ks * SW +
                                           (lane >> 4) * VEC);
          sacc[nt] = mfma_step(qf[ks], kf, sacc[nt], dummy);
        }

      float p[2][4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float mx = -INFINITY;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int key = b * ATT_BKV + nt * 16 + (lane & 15);
          const float sv = key < Skv ? sacc[nt][r] * a.scale_log2 : -INFINITY;
          p[nt][r] = sv;
          mx = fmaxf(mx, sv);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        const float mnew = fmaxf(mrow[r], mx);
        const float alpha = exp2f(mrow[r] - mnew);
        float sum = 0.f;
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          p[nt][r] = exp2f(p[nt][r] - mnew);
          sum += p[nt][r];
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) sum += __shfl_xor(sum, off);
        lrow[r] = lrow[r] * alpha + sum;
        mrow[r] = mnew;
#pragma unroll
        for (int d = 0; d < NOT; ++d) o[d][r] *= alpha;
      }

      // P to LDS (C layout), back in A-operand layout
      float* myP = sP + wave * 16 * PS;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) myP[((lane >> 4) * 4 + r) * PS + nt * 16 + (lane & 15)] = p[nt][r];
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_wave_barrier();

#pragma unroll
      for (int ks = 0; ks < ATT_BKV / SW; ++ks) {
        const float* pr = myP + (lane & 15) * PS + ks * SW + (lane >> 4) * VEC;
        if constexpr (sizeof(T) == 2) {
          uint32_t hi[4], lo[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float x0 = pr[2 * q], x1 = pr[2 * q + 1];
            const uint16_t h0 = f2bf(x0), h1 = f2bf(x1);
            const uint16_t l0 = f2bf(x0 - bf2f(h0)), l1 = f2bf(x1 - bf2f(h1));
            hi[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            lo[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
          }
          const uint4 phi = make_uint4(hi[0], hi[1], hi[2], hi[3]);
          const uint4 plo = make_uint4(lo[0], lo[1], lo[2], lo[3]);
#pragma unroll
          for (int d = 0; d < NOT; ++d) {
            const uint4 vf = *(const uint4*)(sVt + (d * 16 + (lane & 15)) * VS + ks * SW + (lane >> 4) * VEC);
            o[d] = mfma_step(phi, vf, o[d], dummy);
            o[d] = mfma_step(plo, vf, o[d], dummy);
          }
        } else {
          const uint4 pf = make_uint4(__float_as_uint(pr[0]), __float_as_uint(pr[1]),
                                      __float_as_uint(pr[2]), __float_as_uint(pr[3]));
#pragma unroll
          for (int d = 0; d < NOT; ++d) {
            const uint4 vf = *(const uint4*)(sVt + (d * 16 + (lane & 15)) * VS + ks * SW + (lane >> 4) * VEC);
            o[d] = mfma_step(pf, vf, o[d], dummy);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }

    // rows of this lane in the C layout
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rr = (lane >> 4) * 4 + r;
      const int prow = qb * ATT_BQ + wave * 16 + rr;
      if (a.splits == 1) {
        if (prow >= R) continue;
        const int sq = prow / group, h = j * group + prow % group;
        T* op = (T*)a.out + seg * a.seg_o + (size_t)sq * a.ldo + h * a.hd;
        const float inv = 1.f / lrow[r];
#pragma unroll
        for (int d = 0; d < NOT; ++d) {
          const int col = d * 16 + (lane & 15);
          if (col < a.hd) TT<T>::st(op + col, o[d][r] * inv);
        }
      } else {
        const size_t base = ((size_t)work * a.splits + sp) * ATT_BQ + wave * 16 + rr;
#pragma unroll
        for (int d = 0; d < NOT; ++d) a.po[base * HDP + d * 16 + (lane & 15)] = o[d][r];
        if ((lane & 15) == 0) {
          a.pm[base] = mrow[r];
          a.pl[base] = lrow[r];
        }
      }
    }
  }
  VLA_WAVE_END(KK_ATTN);
}

// Merge of the key splits: each thread takes 8 consecutive head dimensions
// of one packed row. The row's maximum over the splits and each split's
// weight 2^(m_s - max) are formed once for the 8 outputs; numerator and
// denominator are summed in split order (splits that saw no key are skipped),
// and the row's 8 outputs go out as one 16-byte store where aligned.
template <typename T, int HDP>
__global__ __launch_bounds__(256) void k_attn_combine(AttnArgs a) {
  VLA_WAVE_BEGIN(KK_ATTN_COMBINE);
  static_assert(HDP % 8 == 0, "8 dimensions per thread");
  constexpr int D8 = HDP / 8;
  const int group = a.nq / a.nkv;
  const int R = a.Sq * group;
  const int nwork = a.qblocks * a.nkv * a.segs;
  const long long total = (long long)nwork * ATT_BQ * D8;
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int d0 = (int)(idx % D8) * 8;
    const long long t = idx / D8;
    const int row = (int)(t % ATT_BQ);
    const int work = (int)(t / ATT_BQ);
    int u = work;
    const int qb = u % a.qblocks;
    u /= a.qblocks;
    const int j = u % a.nkv;
    const int seg = u / a.nkv;
    const int prow = qb * ATT_BQ + row;
    if (prow >= R || d0 >= a.hd) continue;
    float mx = -INFINITY;
    for (int s = 0; s < a.splits; ++s) mx = fmaxf(mx, a.pm[((size_t)work * a.splits + s) * ATT_BQ + row]);
    float num[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, den = 0.f;
    for (int s = 0; s < a.splits; ++s) {
      const size_t base = ((size_t)work * a.splits + s) * ATT_BQ + row;
      const float m = a.pm[base];
      if (m == -INFINITY) continue;
      const float wgt = exp2f(m - mx);
      const float4* po = (const float4*)(a.po + base * HDP + d0);
      const float4 p0 = po[0], p1 = po[1];
      num[0] += wgt * p0.x;
      num[1] += wgt * p0.y;
      num[2] += wgt * p0.z;
      num[3] += wgt * p0.w;
      num[4] += wgt * p1.x;
      num[5] += wgt * p1.y;
      num[6] += wgt * p1.z;
      num[7] += wgt * p1.w;
      den += wgt * a.pl[base];
    }
    const int sq = prow / group, h = j * group + prow % group;
    T* op = (T*)a.out + seg * a.seg_o + (size_t)sq * a.ldo + h * a.hd + d0;
    bool done = false;
    if constexpr (sizeof(T) == 2) {
      if (d0 + 8 <= a.hd && ((uintptr_t)op & 15) == 0) {
        uint16_t o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = f2bf(num[q] / den);
        *(uint4*)op = *(const uint4*)o;
        done = true;
      }
    }
    if (!done)
      for (int q = 0; q < 8 && d0 + q < a.hd; ++q) TT<T>::st(op + q, num[q] / den);
  }
  VLA_WAVE_END(KK_ATTN_COMBINE);
}

static int attn_hdp(int hd, int dtype) {
  const int sw = dtype == DT_BF16 ? 32 : 16;
  int h = (hd + sw - 1) / sw * sw;
  if (h <= 32) return 32;
  if (h <= 64) return 64;
  if (h <= 96) return 96;
  if (h <= 128) return 128;
  if (h <= 256) return 256;
  return -1;
}

static void attn_split(const AttnDesc& d, int* qblocks, int* splits) {
  const int group = d.nq / d.nkv;
  *qblocks = (d.Sq * group + ATT_BQ - 1) / ATT_BQ;
  const int base = *qblocks * d.nkv * (d.plan_segs > 0 ? std::min(d.plan_segs, d.segs) : d.segs);
  const int nblk = (d.S0 + d.S1 + ATT_BKV - 1) / ATT_BKV;
  int s = 1;
  if (base < 128 && nblk >= 4) s = std::min((128 + base - 1) / base, nblk / 2);
  s = std::max(s, 1);
  const int bps = (nblk + s - 1) / s;
  *splits = (nblk + bps - 1) / bps;
}

size_t attn_scratch_floats(const AttnDesc& d) {
  int qb, sp;
  attn_split(d, &qb, &sp);
  if (sp == 1) return 0;
  const int hdp = attn_hdp(d.hd, d.dtype);
  const size_t rows = (size_t)qb * d.nkv * d.segs * sp * ATT_BQ;
  return rows * hdp + 2 * rows;
}

template <typename T, int HDP>
static hipError_t run_attn_t(const AttnArgs& a, const LaunchCaps& caps, hipStream_t st) {
  const int total = a.qblocks * a.nkv * a.segs * a.splits;
  int grid = total;
  if (caps.max_wgs > 0) grid = std::min(grid, caps.max_wgs);
  hipExtLaunchKernelGGL((k_attn<T, HDP>), dim3(grid), dim3(256), 0, st, caps.ev_start,
                        caps.ev_stop, 0, a);
  if (a.splits > 1) {
    const long long n = (long long)a.qblocks * a.nkv * a.segs * ATT_BQ * (HDP / 8);
    int cg = (int)std::min<long long>((n + 255) / 256, 4096);
    if (caps.max_wgs > 0) cg = std::min(cg, caps.max_wgs);
    k_attn_combine<T, HDP><<<cg, 256, 0, st>>>(a);
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t run_attn_hd(const AttnArgs& a, int hdp, const LaunchCaps& caps, hipStream_t st) {
  switch (hdp) {
    case 32: return run_attn_t<T, 32>(a, caps, st);
    case 64: return run_attn_t<T, 64>(a, caps, st);
    case 96: return run_attn_t<T, 96>(a, caps, st);
    case 128: return run_attn_t<T, 128>(a, caps, st);
    case 256: return run_attn_t<T, 256>(a, caps, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention(const AttnDesc& d, const Scratch& s, const LaunchCaps& caps,
                            hipStream_t st) {
  const int hdp = attn_hdp(d.hd, d.dtype);
  if (hdp < 0 || d.nq % d.nkv != 0 || d.S0 + d.S1 <= 0 || d.Sq <= 0) return hipErrorInvalidValue;
  AttnArgs a{};
  a.q = d.q;
  a.k0 = d.k0;
  a.v0 = d.v0;
  a.k1 = d.k1;
  a.v1 = d.v1;
  a.out = d.out;
  a.ldq = d.ldq;
  a.ldkv = d.ldkv;
  a.ldo = d.ldo;
  a.Sq = d.Sq;
  a.nq = d.nq;
  a.nkv = d.nkv;
  a.hd = d.hd;
  a.S0 = d.S0;
  a.S1 = d.S1;
  a.segs = d.segs;
  a.seg_q = d.seg_q;
  a.seg_kv = d.seg_kv;
  a.seg_o = d.seg_o;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.hd));
  attn_split(d, &a.qblocks, &a.splits);
  if (a.splits > 1) {
    const size_t rows = (size_t)a.qblocks * d.nkv * d.segs * a.splits * ATT_BQ;
    if (rows * hdp + 2 * rows > s.floats) return hipErrorInvalidValue;
    a.po = s.ptr;
    a.pm = s.ptr + rows * hdp;
    a.pl = a.pm + rows;
  }
  if (d.dtype == DT_BF16) return run_attn_hd<uint16_t>(a, hdp, caps, st);
  return run_attn_hd<float>(a, hdp, caps, st);
}

// ---------------------------------------------------------------------------
// Attention over the KV cache. K and V sit in MFMA fragment order (see
// kv_kidx / kv_vidx), so every operand load is one contiguous 1 KB per wave
// straight into registers; the 16 packed query rows of a workgroup (row r <->
// query r / group, head r % group of one KV head) are staged once through
// LDS. The key space is [segment 0 padded to a multiple of 32; segment 1
// padded likewise]; keys past a segment's length get a -inf score. The NW
// waves take every NW-th 32-key block, with the next block's K and V
// prefetched into registers.
//
// Everything is computed transposed, so the probabilities never leave the
// registers: S^T = K Q^T puts one query per lane column and keys on the
// rows, and O^T += V^T P^T takes P^T as the B operand straight from the
// score registers (the cache layout puts in each lane group's score rows
// exactly the keys of its B-operand slice). The online softmax is fp32 with
// one running max per query (reduced across the four lane groups) and
// per-lane partial sums, reduced once at the end; P is split into bf16 high
// and remainder parts for the bf16 MFMA. The waves' (max, sum, O) are merged
// through LDS in wave order.
// ---------------------------------------------------------------------------

struct Attn2Args {
  const void* q;
  const void* k0[MAX_FRAMES];  // per frame
  const void* v0[MAX_FRAMES];
  const void* k1;     // frame f: k1 + f k1_blk (elements)
  const void* v1;
  void* out;          // frame f: out + f out_blk
  size_t k1_blk, v1_blk, out_blk;
  int frames;
  int ldq, ldo, out_afrag;
  int Sq, nq, nkv, hd, S0, S1;
  int nb0, nb1;  // 32-key blocks per KV head in each segment's buffers
  int rtiles;    // 16-row tiles of packed rows per KV head
  float scale_log2;
  // key splits: split s of a query tile takes blocks [s bps, (s + 1) bps);
  // with nsplit > 1 its partial (row max, sum, unnormalised O) goes to
  // part and the last split to arrive merges them (see the kernel)
  int nsplit, bps;
  float* part;
  unsigned* cnt;
};

constexpr float ATT_TAU = 8.f;  // lazy-rescaling slack, log2 units
// key splits (attn2_plan): 32-key blocks per wave and split, most splits,
// workgroups beyond which a launch takes no more splits
#ifndef VLA_ATT_BPW
#define VLA_ATT_BPW 4
#endif
constexpr int ATT_BPW = VLA_ATT_BPW;
constexpr int ATT_MAX_SPLITS = 8;
constexpr int ATT_SPLIT_WGS = 512;

// waves per workgroup: eight, or four where a wave needs more than the 256
// registers eight waves leave it
template <typename T, int HDP>
constexpr int att2_waves() {
  return HDP * (int)sizeof(T) >= 512 ? 4 : 8;
}

template <typename T, int HDP, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn2(Attn2Args a) {
  VLA_WAVE_BEGIN(KK_ATTN2);
  constexpr int VEC = 16 / sizeof(T);
  constexpr int SW = 4 * VEC;
  constexpr int NQF = HDP / SW;   // Q fragments (also K fragments per 16-key tile)
  constexpr int NOT = HDP / 16;   // 16-row tiles of O^T
  constexpr int PVS = 32 / SW;    // P V slabs per 32-key block
  constexpr int OS = HDP + 4;     // sO row stride (floats)
  constexpr int QS = HDP + VEC;   // sQ row stride (elements)
  constexpr int NT = 64 * NW;
  constexpr int FRAG = 64 * VEC;  // elements of one 1 KB fragment chunk
  __shared__ __attribute__((aligned(16))) float sO[NW][16 * OS];
  __shared__ float sM[NW][16], sL[NW][16];
  __shared__ __attribute__((aligned(16))) T sQ[16 * QS];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g4 = lane >> 4;  // lane group
  const int group = a.nq / a.nkv;
  const int R = a.Sq * group;
  const int nblk = a.nb0 + a.nb1;
  const int total = a.rtiles * a.nkv;
  const int ns = (a.hd + SW - 1) / SW, ndt = (a.hd + 15) / 16;
  const T dummy = T();
  const Rsrc rq = rsrc(a.q, span(a.Sq * a.frames, a.ldq, a.nq * a.hd, sizeof(T)));

  __shared__ int sLast;
  for (int w = blockIdx.x; w < total * a.frames * a.nsplit; w += gridDim.x) {
    // item w: split sp of query tile wt; frame f: its queries, its two key
    // segments and its output block
    const int sp = w % a.nsplit, wt = w / a.nsplit;
    const int f = __builtin_amdgcn_readfirstlane(wt / total), wl = wt % total;
    const int b_lo = sp * a.bps, b_hi = min(nblk, b_lo + a.bps);
    const int rt = wl % a.rtiles, j = wl / a.rtiles;
    const Rsrc rk0 = rsrc(a.k0[f], (size_t)a.nkv * a.nb0 * 2 * ns * FRAG * sizeof(T));
    const Rsrc rv0 = rsrc(a.v0[f], (size_t)a.nkv * a.nb0 * ndt * PVS * FRAG * sizeof(T));
    const Rsrc rk1 = rsrc(a.k1 ? (const T*)a.k1 + f * a.k1_blk : a.k0[f],
                          a.k1 ? (size_t)a.nkv * a.nb1 * 2 * ns * FRAG * sizeof(T) : 0);
    const Rsrc rv1 = rsrc(a.v1 ? (const T*)a.v1 + f * a.v1_blk : a.v0[f],
                          a.v1 ? (size_t)a.nkv * a.nb1 * ndt * PVS * FRAG * sizeof(T) : 0);

    // the workgroup's 16 packed query rows, row-contiguous loads (issued
    // before K and V so that waiting for them does not wait for K and V)
    constexpr int QCH = 16 * (HDP / VEC), QPT = (QCH + NT - 1) / NT;
    uint4 qld[QPT];
#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int c = tid + u * NT;
      const int rr = c / (HDP / VEC), d = (c % (HDP / VEC)) * VEC;
      const int r = rt * 16 + rr;
      const int sq = f * a.Sq + r / group, h = j * group + r % group;
      const bool ok = c < QCH && r < R && d < a.hd;
      qld[u] = bld16(rq, ok ? (uint32_t)(((size_t)sq * a.ldq + h * a.hd + d) * sizeof(T)) : OOB);
    }

    // fragment loads of one 32-key block (b past the split's end reads zeros)
    auto load_k = [&](int b, uint4 (&kf)[2][NQF]) {
      const bool seg1 = b >= a.nb0;
      const int bl = seg1 ? b - a.nb0 : b, nb = seg1 ? a.nb1 : a.nb0;
      const Rsrc rk = seg1 ? rk1 : rk0;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int ks = 0; ks < NQF; ++ks) {
          const bool ok = b < b_hi && ks * SW + g4 * VEC < a.hd;
          const size_t off = ((((size_t)j * nb + bl) * 2 + nt) * ns + ks) * FRAG + lane * VEC;
          kf[nt][ks] = bld16(rk, ok ? (uint32_t)(off * sizeof(T)) : OOB);
        }
    };
    auto load_v = [&](int b, uint4 (&vf)[NOT][PVS]) {
      const bool seg1 = b >= a.nb0;
      const int bl = seg1 ? b - a.nb0 : b, nb = seg1 ? a.nb1 : a.nb0;
      const Rsrc rv = seg1 ? rv1 : rv0;
#pragma unroll
      for (int dt = 0; dt < NOT; ++dt)
#pragma unroll
        for (int kk = 0; kk < PVS; ++kk) {
          const bool ok = b < b_hi && dt * 16 + (lane & 15) < a.hd;
          const size_t off = ((((size_t)j * nb + bl) * ndt + dt) * PVS + kk) * FRAG + lane * VEC;
          vf[dt][kk] = bld16(rv, ok ? (uint32_t)(off * sizeof(T)) : OOB);
        }
    };

    // Loads are issued unconditionally: with the same loads in flight on
    // every path each wait covers only the oldest group.
    uint4 kf[2][NQF], vf[NOT][PVS];
    load_k(b_lo + wave, kf);
    load_v(b_lo + wave, vf);

    float mrun = -INFINITY, lpart = 0.f;  // running max of this lane's query; partial sum
    f32x4 o[NOT];
#pragma unroll
    for (int d = 0; d < NOT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int u = 0; u < QPT; ++u) {
      const int c = tid + u * NT;
      if (c < QCH) *(uint4*)&sQ[(c / (HDP / VEC)) * QS + (c % (HDP / VEC)) * VEC] = qld[u];
    }
    __syncthreads();
    // Q^T as the B operand: lane column = packed row, 16-byte slice of d
    uint4 qf[NQF];
#pragma unroll
    for (int ks = 0; ks < NQF; ++ks) qf[ks] = *(const uint4*)&sQ[(lane & 15) * QS + ks * SW + g4 * VEC];

    auto process = [&](int b) {
      const bool seg1 = b >= a.nb0;
      const int kloc = (seg1 ? b - a.nb0 : b) * 32;
      const int slen = seg1 ? a.S1 : a.S0;
      // S^T for 32 keys x 16 queries, two accumulators per tile
      f32x4 sacc[2][2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) sacc[nt][0] = sacc[nt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < NQF; ++ks)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) sacc[nt][ks & 1] = mfma_step(kf[nt][ks], qf[ks], sacc[nt][ks & 1], dummy);
      load_k(b + NW, kf);
      float p[2][4];
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          // key of score row 4 g4 + r in tile nt (the cache layout's order)
          const int kin = sizeof(T) == 2 ? 8 * g4 + 4 * nt + r : 16 * nt + 4 * g4 + r;
          const float sv = kloc + kin < slen ? (sacc[nt][0][r] + sacc[nt][1][r]) * a.scale_log2 : -INFINITY;
          p[nt][r] = sv;
          mx = fmaxf(mx, sv);
        }
      mx = wave_max_x16_x32(mx);
      // Lazy rescaling: the reference point mrun only moves when a score
      // exceeds it by more than 2^ATT_TAU (or on the first finite score), so
      // the O rescale is skipped for most blocks; probabilities stay below
      // 2^ATT_TAU and the final normalisation is unchanged.
      const bool move = mx > mrun + ATT_TAU;
      if (__any(move)) {
        const float mnew = move ? mx : mrun;
        const float alpha = mrun == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mrun - mnew);
        lpart *= alpha;
#pragma unroll
        for (int d = 0; d < NOT; ++d) o[d] *= alpha;
        mrun = mnew;
      }
      float sum = 0.f;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          p[nt][r] = p[nt][r] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(p[nt][r] - mrun);
          sum += p[nt][r];
        }
      lpart += sum;
      if constexpr (sizeof(T) == 2) {
        // P^T slice of lane group g4: keys 8 g4 .. 8 g4 + 7 = rows 4 g4 + r of tiles 0, 1
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float x0 = p[q >> 1][2 * (q & 1)], x1 = p[q >> 1][2 * (q & 1) + 1];
          hi[q] = f2bf2(x0, x1);
          lo[q] = f2bf2(x0 - bf2f((uint16_t)hi[q]), x1 - bf2f((uint16_t)(hi[q] >> 16)));
        }
        const uint4 phi = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        const uint4 plo = make_uint4(lo[0], lo[1], lo[2], lo[3]);
#pragma unroll
        for (int d = 0; d < NOT; ++d) {
          o[d] = mfma_step(vf[d][0], phi, o[d], dummy);
          o[d] = mfma_step(vf[d][0], plo, o[d], dummy);
        }
      } else {
        // slab kk = tile kk: keys 16 kk + 4 g4 .. + 3
#pragma unroll
        for (int kk = 0; kk < PVS; ++kk) {
          const uint4 pf = make_uint4(__float_as_uint(p[kk][0]), __float_as_uint(p[kk][1]),
                                      __float_as_uint(p[kk][2]), __float_as_uint(p[kk][3]));
#pragma unroll
          for (int d = 0; d < NOT; ++d) o[d] = mfma_step(vf[d][kk], pf, o[d], dummy);
        }
      }
      load_v(b + NW, vf);
    };

    for (int b = b_lo + wave; b < b_hi; b += NW) process(b);

    // the four lane groups' partial sums of one query
    lpart = wave_sum_x16_x32(lpart);
    // O^T registers: lane column = packed row (lane & 15), rows d = 16 dt + 4 g4 + r
#pragma unroll
    for (int d = 0; d < NOT; ++d)
      *(f32x4*)&sO[wave][(lane & 15) * OS + d * 16 + 4 * g4] = o[d];
    if (g4 == 0) {
      sM[wave][lane] = mrun;
      sL[wave][lane] = lpart;
    }
    __syncthreads();
    // merge the waves in order; eight consecutive outputs per thread
    constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
    auto store_out = [&](int prow, int d0, const float (&num)[8], float den) {
      const float inv = 1.f / den;
      const int sq = prow / group, col = (j * group + prow % group) * a.hd + d0;
      // 16-byte pieces: one VEC group each in the row-block operand layout
      auto at = [&](int c) {
        return (T*)a.out + f * a.out_blk + (a.out_afrag ? afrag_index(DT, sq, c) : (size_t)sq * a.ldo + c);
      };
      if constexpr (sizeof(T) == 2) {
        uint32_t pk[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) pk[e] = f2bf2(num[2 * e] * inv, num[2 * e + 1] * inv);
        *(uint4*)at(col) = make_uint4(pk[0], pk[1], pk[2], pk[3]);
      } else {
        *(float4*)at(col) = make_float4(num[0] * inv, num[1] * inv, num[2] * inv, num[3] * inv);
        *(float4*)at(col + 4) = make_float4(num[4] * inv, num[5] * inv, num[6] * inv, num[7] * inv);
      }
    };
    // a split's partial: [16 rows][HDP] unnormalised O, then 16 row maxima
    // and 16 sums
    constexpr int PSZ = 16 * HDP + 32;
    const Rsrc rp = rsrc(a.part, a.nsplit > 1 ? (size_t)total * a.frames * a.nsplit * PSZ * sizeof(float) : 0);
    const uint32_t mybase = (uint32_t)(((size_t)wt * a.nsplit + sp) * PSZ);
    for (int idx = tid * 8; idx < 16 * HDP; idx += NT * 8) {
      const int rr = idx / HDP, d0 = idx % HDP;
      const int prow = rt * 16 + rr;
      if (prow >= R || d0 >= a.hd) continue;
      float mx = -INFINITY;
#pragma unroll
      for (int u = 0; u < NW; ++u) mx = fmaxf(mx, sM[u][rr]);
      float num[8], den = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) num[e] = 0.f;
#pragma unroll
      for (int u = 0; u < NW; ++u) {
        const float wgt = sM[u][rr] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sM[u][rr] - mx);
        const f32x4 v0 = *(const f32x4*)&sO[u][rr * OS + d0];
        const f32x4 v1 = *(const f32x4*)&sO[u][rr * OS + d0 + 4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          num[e] += wgt * v0[e];
          num[4 + e] += wgt * v1[e];
        }
        den += wgt * sL[u][rr];
      }
      if (a.nsplit == 1) {
        store_out(prow, d0, num, den);
      } else {
        const uint32_t o = (mybase + rr * HDP + d0) * 4;
        bst16_sc1(rp, o, f32x4{num[0], num[1], num[2], num[3]});
        bst16_sc1(rp, o + 16, f32x4{num[4], num[5], num[6], num[7]});
        if (d0 == 0) {
          bst1_sc1(rp, (mybase + 16 * HDP + rr) * 4, mx);
          bst1_sc1(rp, (mybase + 16 * HDP + 16 + rr) * 4, den);
        }
      }
    }
    if (a.nsplit > 1) {
      // Every thread's partial stores have completed (vmcnt counts stores
      // on this architecture) before thread 0 counts this split in; the
      // split that counts last sees every other split's stores done and
      // merges. No split waits for another: the last arrival does the work.
      __builtin_amdgcn_s_waitcnt(VMCNT0);
      __syncthreads();
      if (tid == 0) {
        const unsigned old = __hip_atomic_fetch_add(a.cnt + wt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sLast = old == (unsigned)(a.nsplit - 1);
        // the counter goes back to zero for the next launch (and graph replay)
        if (sLast) __hip_atomic_store(a.cnt + wt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();
      if (sLast) {
        const uint32_t tile = (uint32_t)((size_t)wt * a.nsplit * PSZ);
        for (int idx = tid * 8; idx < 16 * HDP; idx += NT * 8) {
          const int rr = idx / HDP, d0 = idx % HDP;
          const int prow = rt * 16 + rr;
          if (prow >= R || d0 >= a.hd) continue;
          // every split's values in flight at once; splits past nsplit read
          // zeros and are skipped below
          float mq[ATT_MAX_SPLITS], lq[ATT_MAX_SPLITS];
          f32x4 oq[ATT_MAX_SPLITS][2];
#pragma unroll
          for (int q = 0; q < ATT_MAX_SPLITS; ++q) {
            const bool ok = q < a.nsplit;
            const uint32_t b = tile + q * PSZ;
            oq[q][0] = bld16_sc1(rp, ok ? (b + rr * HDP + d0) * 4 : OOB);
            oq[q][1] = bld16_sc1(rp, ok ? (b + rr * HDP + d0 + 4) * 4 : OOB);
            mq[q] = bld1_sc1(rp, ok ? (b + 16 * HDP + rr) * 4 : OOB);
            lq[q] = bld1_sc1(rp, ok ? (b + 16 * HDP + 16 + rr) * 4 : OOB);
          }
          // splits in order: the result does not depend on the arrival order
          float mx = -INFINITY;
#pragma unroll
          for (int q = 0; q < ATT_MAX_SPLITS; ++q)
            if (q < a.nsplit) mx = fmaxf(mx, mq[q]);
          float num[8], den = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) num[e] = 0.f;
#pragma unroll
          for (int q = 0; q < ATT_MAX_SPLITS; ++q) {
            if (q >= a.nsplit) continue;
            const float wgt = mq[q] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mq[q] - mx);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              num[e] += wgt * oq[q][0][e];
              num[4 + e] += wgt * oq[q][1][e];
            }
            den += wgt * lq[q];
          }
          store_out(prow, d0, num, den);
        }
      }
    }
    __syncthreads();
  }
  VLA_WAVE_END(KK_ATTN2);
}

// Key splits of the cache attention. A split gives each wave ATT_BPW 32-key
// blocks; there are at most ATT_MAX_SPLITS of them, and splits stop where the
// launch would exceed ATT_SPLIT_WGS workgroups (enough query tiles fill the
// chip without them). Returns the split count and the blocks per split.
static int attn2_plan(int nblk, int nw, int tiles, int* bps) {
  int ns = std::min((nblk + nw * ATT_BPW - 1) / (nw * ATT_BPW), ATT_MAX_SPLITS);
  while (ns > 1 && tiles * ns > ATT_SPLIT_WGS) --ns;
  if (ns <= 1) {
    *bps = nblk;
    return 1;
  }
  // balanced splits of whole wave rounds
  const int per = (nblk + ns - 1) / ns;
  *bps = (per + nw - 1) / nw * nw;
  return (nblk + *bps - 1) / *bps;
}

// a launch uses splits only when the caller gave room for their partials and
// counters (otherwise one split, the whole key range)
template <typename T, int H>
static void attn2_split(Attn2Args& a, float* part, size_t part_floats, unsigned* cnt, int cnt_n) {
  const int nblk = a.nb0 + a.nb1;
  const int tiles = a.rtiles * a.nkv * a.frames;
  int bps;
  int ns = attn2_plan(nblk, att2_waves<T, H>(), tiles, &bps);
  if (ns > 1 && (!part || !cnt || cnt_n < tiles || (size_t)tiles * ns * (16 * H + 32) > part_floats)) ns = 1;
  a.nsplit = ns;
  a.bps = ns > 1 ? bps : nblk;
  a.part = part;
  a.cnt = cnt;
}

template <typename T>
static hipError_t run_attn2_t(Attn2Args& a, int hdp, const LaunchCaps& caps, hipStream_t st, float* part,
                              size_t part_floats, unsigned* cnt, int cnt_n) {
  if (sizeof(T) == 4 && hdp > 128) return hipErrorInvalidValue;  // fp32: head dim <= 128
  switch (hdp) {
    case 32: attn2_split<T, 32>(a, part, part_floats, cnt, cnt_n); break;
    case 64: attn2_split<T, 64>(a, part, part_floats, cnt, cnt_n); break;
    case 96: attn2_split<T, 96>(a, part, part_floats, cnt, cnt_n); break;
    case 128: attn2_split<T, 128>(a, part, part_floats, cnt, cnt_n); break;
    case 256: attn2_split<T, 256>(a, part, part_floats, cnt, cnt_n); break;
    default: return hipErrorInvalidValue;
  }
  int grid = a.rtiles * a.nkv * a.frames * a.nsplit;
  if (caps.max_wgs > 0) grid = std::min(grid, caps.max_wgs);
#define VLA_ATTN2(H)                                                                           \
  hipExtLaunchKernelGGL((k_attn2<T, H, att2_waves<T, H>()>), dim3(grid),                        \
                        dim3(64 * att2_waves<T, H>()), 0, st, caps.ev_start, caps.ev_stop, 0, a)
  switch (hdp) {
    case 32: VLA_ATTN2(32); break;
    case 64: VLA_ATTN2(64); break;
    case 96: VLA_ATTN2(96); break;
    case 128: VLA_ATTN2(128); break;
    case 256:
      if constexpr (sizeof(T) == 2) VLA_ATTN2(256);
      break;
    default: return hipErrorInvalidValue;
  }
#undef VLA_ATTN2
  return hipGetLastError();
}

hipError_t launch_attention_kv(const AttnKvDesc& d, const LaunchCaps& caps, hipStream_t st) {
  const int hdp = attn_hdp(d.hd, d.dtype);
  if (hdp < 0 || d.nq % d.nkv != 0 || d.S0 <= 0 || d.S1 < 0 || d.Sq <= 0 ||
      (d.S1 > 0 && (!d.k1 || !d.v1)) || d.hd % 8 != 0 || (d.out_afrag && d.Sq > 64) ||
      (!d.out_afrag && ((size_t)d.ldo * (d.dtype == DT_BF16 ? 2 : 4)) % 16 != 0) ||
      ((uintptr_t)d.out & 15) != 0 || d.frames < 1 || d.frames > MAX_FRAMES ||
      (d.frames > 1 && (d.out_blk * (d.dtype == DT_BF16 ? 2 : 4)) % 16 != 0))
    return hipErrorInvalidValue;
  for (int f = 1; f < d.frames; ++f)
    if (!d.k0f[f] || !d.v0f[f]) return hipErrorInvalidValue;
  Attn2Args a{};
  a.q = d.q;
  a.k0[0] = d.k0;
  a.v0[0] = d.v0;
  for (int f = 1; f < MAX_FRAMES; ++f) {
    a.k0[f] = f < d.frames ? d.k0f[f] : d.k0;
    a.v0[f] = f < d.frames ? d.v0f[f] : d.v0;
  }
  a.k1 = d.S1 > 0 ? d.k1 : nullptr;
  a.v1 = d.S1 > 0 ? d.v1 : nullptr;
  a.k1_blk = d.k1_blk;
  a.v1_blk = d.v1_blk;
  a.out_blk = d.out_blk;
  a.frames = d.frames;
  a.out = d.out;
  a.ldq = d.ldq;
  a.ldo = d.ldo;
  a.out_afrag = d.out_afrag;
  a.Sq = d.Sq;
  a.nq = d.nq;
  a.nkv = d.nkv;
  a.hd = d.hd;
  a.S0 = d.S0;
  a.S1 = d.S1;
  a.nb0 = (d.S0 + 31) / 32;
  a.nb1 = (d.S1 + 31) / 32;
  a.rtiles = (d.Sq * (d.nq / d.nkv) + 15) / 16;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.hd));
  if (d.dtype == DT_BF16) return run_attn2_t<uint16_t>(a, hdp, caps, st, d.part, d.part_floats, d.cnt, d.cnt_n);
  return run_attn2_t<float>(a, hdp, caps, st, d.part, d.part_floats, d.cnt, d.cnt_n);
}

size_t attn_kv_split_floats(int dtype, int frames, int Sq, int nq, int nkv, int hd, int S0, int S1, int* counters) {
  const int hdp = attn_hdp(hd, dtype);
  *counters = 0;
  if (hdp < 0 || nkv <= 0 || nq % nkv) return 0;
  const int nw = dtype == DT_BF16 ? (hdp * 2 >= 512 ? 4 : 8) : (hdp * 4 >= 512 ? 4 : 8);
  const int nblk = (S0 + 31) / 32 + (S1 + 31) / 32;
  const int tiles = (Sq * (nq / nkv) + 15) / 16 * nkv * frames;
  int bps;
  const int ns = attn2_plan(nblk, nw, tiles, &bps);
  *counters = ns > 1 ? tiles : 0;
  return ns > 1 ? (size_t)tiles * ns * (16 * hdp + 32) : 0;
}

// ---------------------------------------------------------------------------
// Row norms (LayerNorm with biased variance, or RMSNorm), fp32 statistics,
// one workgroup per row, fixed-order tree reduction.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// One workgroup per row. Thread t owns the four-column groups starting at
// columns 4 t, 4 t + 1024, ... (16-byte accesses), and every load of the row
// (x, the split partials, bias, column scale, gain and shift) is issued before
// the first use, so a row costs one memory round trip.
constexpr int NORM_VPT = 2;  // four-column groups per thread: d <= 2048


template <typename T>
__global__ __launch_bounds__(256) void k_norm(NormDesc n) {
  VLA_WAVE_BEGIN(KK_NORM);
  constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
  constexpr int SPL = 8;  // split partials requested together
  __shared__ float red[4];
  const int rows = n.rows, d = n.d, ldx = n.ldx, splits = n.splits;
  float* __restrict__ x = n.x;
  const size_t pstride = (size_t)rows * d;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f}, one4 = {1.f, 1.f, 1.f, 1.f};
  // absent vectors get an empty range: their loads return zeros
  const Rsrc rx = rsrc(x, span(rows, ldx, d, 4));
  const Rsrc rp = rsrc(n.part ? n.part : x, n.part ? (size_t)splits * pstride * 4 : 0);
  const Rsrc rb = rsrc(n.bias ? n.bias : x, n.bias ? (size_t)d * 4 : 0);
  const Rsrc rc = rsrc(n.colscale ? n.colscale : x, n.colscale ? (size_t)d * 4 : 0);
  const Rsrc rg = rsrc(n.g, (size_t)d * 4);
  const Rsrc rs = rsrc(n.b ? n.b : x, n.b ? (size_t)d * 4 : 0);
  for (int row = blockIdx.x; row < rows; row += gridDim.x) {
    f32x4 v[NORM_VPT], add[NORM_VPT], cs[NORM_VPT], gn[NORM_VPT], sh[NORM_VPT];
#pragma unroll
    for (int q = 0; q < NORM_VPT; ++q) {
      const int c = (threadIdx.x + q * 256) * 4;
      const bool ok = c < d;
      v[q] = bld4f(rx, ok ? (uint32_t)(((size_t)row * ldx + c) * 4) : OOB);
      add[q] = bld4f(rb, ok ? (uint32_t)(c * 4) : OOB);
      cs[q] = bld4f(rc, ok ? (uint32_t)(c * 4) : OOB);
      gn[q] = bld4f(rg, ok ? (uint32_t)(c * 4) : OOB);
      sh[q] = bld4f(rs, ok ? (uint32_t)(c * 4) : OOB);
    }
    if (splits > 0) {
      // partials summed in split order, SPL splits' loads in flight at once
      f32x4 sum[NORM_VPT];
#pragma unroll
      for (int q = 0; q < NORM_VPT; ++q) sum[q] = zero4;
      for (int sp = 0; sp < splits; sp += SPL) {
        f32x4 t[SPL][NORM_VPT];
#pragma unroll
        for (int u = 0; u < SPL; ++u)
#pragma unroll
          for (int q = 0; q < NORM_VPT; ++q) {
            const int c = (threadIdx.x + q * 256) * 4;
            const bool ok = c < d && sp + u < splits;
            t[u][q] = bld4f(rp, ok ? (uint32_t)(((size_t)row * d + (sp + u) * pstride + c) * 4) : OOB);
          }
#pragma unroll
        for (int u = 0; u < SPL; ++u)
#pragma unroll
          for (int q = 0; q < NORM_VPT; ++q)
            if (sp + u < splits) sum[q] += t[u][q];
      }
#pragma unroll
      for (int q = 0; q < NORM_VPT; ++q) add[q] += n.colscale ? cs[q] * sum[q] : sum[q];
    }
    float s1 = 0.f;
#pragma unroll
    for (int q = 0; q < NORM_VPT; ++q) {
      const int c = (threadIdx.x + q * 256) * 4;
      if (c < d) {
        if (splits > 0) {
          v[q] += add[q];
          *(f32x4*)(x + (size_t)row * ldx + c) = v[q];
        }
        s1 += (v[q][0] + v[q][1]) + (v[q][2] + v[q][3]);
      }
    }
    const float mean = n.rms ? 0.f : block_sum(s1, red) / d;
    float s2 = 0.f;
#pragma unroll
    for (int q = 0; q < NORM_VPT; ++q) {
      const int c = (threadIdx.x + q * 256) * 4;
      if (c < d) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float cd = v[q][e] - mean;
          s2 += cd * cd;
        }
      }
    }
    const float inv = 1.f / sqrtf(block_sum(s2, red) / d + 1e-6f);
    // output row and column offset (pixel shuffle moves whole rows)
    size_t obase = (size_t)row * n.ldo;
    if (n.shuffle > 1) {
      const int s = n.shuffle, view = row / n.tview, t = row % n.tview;
      const int y = t / n.grid_w, xx = t % n.grid_w;
      const int orow = view * (n.tview / (s * s)) + (y / s) * (n.grid_w / s) + xx / s;
      obase = (size_t)orow * n.ldo + (size_t)((y % s) * s + xx % s) * d;
    }
#pragma unroll
    for (int q = 0; q < NORM_VPT; ++q) {
      const int c = (threadIdx.x + q * 256) * 4;
      if (c < d) {
        const f32x4 gi = n.g_plus_one ? one4 + gn[q] : gn[q];
        f32x4 y = (v[q] - mean) * inv * gi;
        if (n.b) y += sh[q];
        // four consecutive columns are contiguous in both output layouts
        T* dst = (T*)n.out + (n.afrag ? afrag_index_blk(DT, row, c, n.blk_rows, n.blk_out) : obase + c);
        if constexpr (sizeof(T) == 2)
          *(uint2*)dst = make_uint2(f2bf2(y[0], y[1]), f2bf2(y[2], y[3]));
        else
          *(f32x4*)dst = y;
      }
    }
  }
  VLA_WAVE_END(KK_NORM);
}

// Rows of at most 1024 columns (the action expert's): one wave per row, four
// rows per workgroup. Lane l owns the four-column groups starting at columns
// 4 l, 4 l + 256, 4 l + 512 and 4 l + 768; every load of the row is issued
// before the first use, the split partials are added in split order as in
// k_norm, and the row statistics are reduced inside the wave (no LDS round
// trip, no barrier), which shortens the launch for the many small norms of
// the action loop. (The column sums are grouped differently from k_norm's,
// so a row's statistics may differ from it in the last bits.)
constexpr int NORMW_VPL = 4;  // four-column groups per lane: d <= 1024
template <typename T>
__global__ __launch_bounds__(256) void k_norm_w(NormDesc n) {
  VLA_WAVE_BEGIN(KK_NORM);
  constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
  constexpr int SPL = 4;  // split partials requested together
  const int rows = n.rows, d = n.d, ldx = n.ldx, splits = n.splits;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float* __restrict__ x = n.x;
  const size_t pstride = (size_t)rows * d;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f}, one4 = {1.f, 1.f, 1.f, 1.f};
  const Rsrc rx = rsrc(x, span(rows, ldx, d, 4));
  const Rsrc rp = rsrc(n.part ? n.part : x, n.part ? (size_t)splits * pstride * 4 : 0);
  const Rsrc rb = rsrc(n.bias ? n.bias : x, n.bias ? (size_t)d * 4 : 0);
  const Rsrc rc = rsrc(n.colscale ? n.colscale : x, n.colscale ? (size_t)d * 4 : 0);
  const Rsrc rg = rsrc(n.g, (size_t)d * 4);
  const Rsrc rs = rsrc(n.b ? n.b : x, n.b ? (size_t)d * 4 : 0);
  for (int row = blockIdx.x * 4 + wave; row < rows; row += gridDim.x * 4) {
    f32x4 v[NORMW_VPL], add[NORMW_VPL], cs[NORMW_VPL], gn[NORMW_VPL], sh[NORMW_VPL];
#pragma unroll
    for (int q = 0; q < NORMW_VPL; ++q) {
      const int c = (lane + q * 64) * 4;
      const bool ok = c < d;
      v[q] = bld4f(rx, ok ? (uint32_t)(((size_t)row * ldx + c) * 4) : OOB);
      add[q] = bld4f(rb, ok ? (uint32_t)(c * 4) : OOB);
      cs[q] = bld4f(rc, ok ? (uint32_t)(c * 4) : OOB);
      gn[q] = bld4f(rg, ok ? (uint32_t)(c * 4) : OOB);
      sh[q] = bld4f(rs, ok ? (uint32_t)(c * 4) : OOB);
    }
    if (splits > 0) {
      f32x4 sum[NORMW_VPL];
#pragma unroll
      for (int q = 0; q < NORMW_VPL; ++q) sum[q] = zero4;
      for (int sp = 0; sp < splits; sp += SPL) {
        f32x4 t[SPL][NORMW_VPL];
#pragma unroll
        for (int u = 0; u < SPL; ++u)
#pragma unroll
          for (int q = 0; q < NORMW_VPL; ++q) {
            const int c = (lane + q * 64) * 4;
            const bool ok = c < d && sp + u < splits;
            t[u][q] = bld4f(rp, ok ? (uint32_t)(((size_t)row * d + (sp + u) * pstride + c) * 4) : OOB);
          }
#pragma unroll
        for (int u = 0; u < SPL; ++u)
#pragma unroll
          for (int q = 0; q < NORMW_VPL; ++q)
            if (sp + u < splits) sum[q] += t[u][q];
      }
#pragma unroll
      for (int q = 0; q < NORMW_VPL; ++q) add[q] += n.colscale ? cs[q] * sum[q] : sum[q];
    }
    float s1 = 0.f;
#pragma unroll
    for (int q = 0; q < NORMW_VPL; ++q) {
      const int c = (lane + q * 64) * 4;
      if (c < d) {
        if (splits > 0) {
          v[q] += add[q];
          *(f32x4*)(x + (size_t)row * ldx + c) = v[q];
        }
        s1 += (v[q][0] + v[q][1]) + (v[q][2] + v[q][3]);
      }
    }
    float mean = 0.f;
    if (!n.rms) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) s1 += __shfl_xor(s1, off);
      mean = s1 / d;
    }
    float s2 = 0.f;
#pragma unroll
    for (int q = 0; q < NORMW_VPL; ++q) {
      const int c = (lane + q * 64) * 4;
      if (c < d) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float cd = v[q][e] - mean;
          s2 += cd * cd;
        }
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s2 += __shfl_xor(s2, off);
    const float inv = 1.f / sqrtf(s2 / d + 1e-6f);
#pragma unroll
    for (int q = 0; q < NORMW_VPL; ++q) {
      const int c = (lane + q * 64) * 4;
      if (c < d) {
        const f32x4 gi = n.g_plus_one ? one4 + gn[q] : gn[q];
        f32x4 y = (v[q] - mean) * inv * gi;
        if (n.b) y += sh[q];
        T* dst = (T*)n.out + (n.afrag ? afrag_index_blk(DT, row, c, n.blk_rows, n.blk_out) : (size_t)row * n.ldo + c);
        if constexpr (sizeof(T) == 2)
          *(uint2*)dst = make_uint2(f2bf2(y[0], y[1]), f2bf2(y[2], y[3]));
        else
          *(f32x4*)dst = y;
      }
    }
  }
  VLA_WAVE_END(KK_NORM);
}

hipError_t launch_norm(const NormDesc& n, hipStream_t st) {
  // four-column accesses: 16-byte fp32 loads and stores, 8-byte bf16 stores
  auto mis = [](const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) != 0; };
  if (mis(n.x, 16) || mis(n.part, 16) || mis(n.bias, 16) || mis(n.colscale, 16) ||
      mis(n.g, 16) || mis(n.b, 16) || mis(n.out, n.dtype == DT_BF16 ? 8 : 16))
    return hipErrorInvalidValue;
  if (n.d > 1024 * NORM_VPT || n.d % 4 || n.ldx % 4 || (!n.afrag && n.ldo % 4) ||
      (n.afrag && (n.blk_rows > 0 ? n.blk_rows > 64 : n.rows > 64)) || !n.x || !n.g || !n.out ||
      (n.shuffle > 1 && (n.grid_w % n.shuffle || n.tview % (n.shuffle * n.grid_w) || n.afrag)))
    return hipErrorInvalidValue;
  if (n.d <= 256 * NORMW_VPL && n.shuffle <= 1) {  // a wave per row
    const int grid = std::min((n.rows + 3) / 4, 4096);
    if (n.dtype == DT_BF16)
      k_norm_w<uint16_t><<<grid, 256, 0, st>>>(n);
    else
      k_norm_w<float><<<grid, 256, 0, st>>>(n);
    return hipGetLastError();
  }
  const int grid = std::min(n.rows, 4096);
  if (n.dtype == DT_BF16)
    k_norm<uint16_t><<<grid, 256, 0, st>>>(n);
  else
    k_norm<float><<<grid, 256, 0, st>>>(n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Small gathers
// ---------------------------------------------------------------------------

template <typename T>
__global__ void k_patchify(const float* __restrict__ pix, int views, int H, int W, int p,
                           T* __restrict__ out, int ldo) {
  VLA_WAVE_BEGIN(KK_PATCHIFY);
  const int gw = W / p, gh = H / p, T_ = gh * gw, kp = 3 * p * p;
  const long long total = (long long)views * T_ * ldo;
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % ldo);
    const long long row = idx / ldo;
    float v = 0.f;
    if (c < kp) {
      const int view = (int)(row / T_), t = (int)(row % T_);
      const int pi = t / gw, pj = t % gw;
      const int ch = c % 3, rc = c / 3, pr = rc / p, pc = rc % p;
      v = pix[(((size_t)view * H + pi * p + pr) * W + pj * p + pc) * 3 + ch];
    }
    TT<T>::st(out + idx, v);
  }
  VLA_WAVE_END(KK_PATCHIFY);
}

hipError_t launch_patchify(int dtype, const float* pix, int views, int H, int W, int p, void* out,
                           int ldo, hipStream_t st) {
  const long long total = (long long)views * (H / p) * (W / p) * ldo;
  const int grid = (int)std::min<long long>((total + 255) / 256, 4096);
  if (dtype == DT_BF16)
    k_patchify<uint16_t><<<grid, 256, 0, st>>>(pix, views, H, W, p, (uint16_t*)out, ldo);
  else
    k_patchify<float><<<grid, 256, 0, st>>>(pix, views, H, W, p, (float*)out, ldo);
  return hipGetLastError();
}

template <typename T>
__global__ void k_embed(const T* __restrict__ E, int d, int vocab, const int32_t* __restrict__ ids,
                        int n, float scale, float* __restrict__ x, int ldx) {
  VLA_WAVE_BEGIN(KK_EMBED);
  for (int row = blockIdx.x; row < n; row += gridDim.x) {
    const int id = min(max(ids[row], 0), vocab - 1);  // out-of-range ids are clamped
    const T* er = E + (size_t)id * d;
    for (int i = threadIdx.x; i < d; i += blockDim.x) x[(size_t)row * ldx + i] = TT<T>::ld(er + i) * scale;
  }
  VLA_WAVE_END(KK_EMBED);
}

hipError_t launch_embed(int dtype, const void* E, int d, int vocab, const int32_t* ids, int n,
                        float scale, float* x, int ldx, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int grid = std::min(n, 1024);
  if (dtype == DT_BF16)
    k_embed<uint16_t><<<grid, 256, 0, st>>>((const uint16_t*)E, d, vocab, ids, n, scale, x, ldx);
  else
    k_embed<float><<<grid, 256, 0, st>>>((const float*)E, d, vocab, ids, n, scale, x, ldx);
  return hipGetLastError();
}

template <typename T>
__global__ void k_cvt_pad(const float* __restrict__ src, int rows, int cols, T* __restrict__ dst,
                          int ld, int afrag, float* __restrict__ dst32, int blk_rows, size_t blk_elems) {
  VLA_WAVE_BEGIN(KK_CVT);
  constexpr int DT = sizeof(T) == 2 ? DT_BF16 : DT_F32;
  const long long total = (long long)rows * ld;
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % ld);
    const long long r = idx / ld;
    const float v = c < cols ? src[r * cols + c] : 0.f;
    TT<T>::st(dst + (afrag ? afrag_index_blk(DT, (int)r, c, blk_rows, blk_elems) : (size_t)idx), v);
    if (dst32 && c < cols) dst32[r * cols + c] = v;
  }
  VLA_WAVE_END(KK_CVT);
}

hipError_t launch_cvt_pad(int dtype, const float* src, int rows, int cols, void* dst, int ld_dst,
                          bool afrag, float* dst_f32, hipStream_t st, int blk_rows, size_t blk_elems) {
  if (afrag && (blk_rows > 0 ? blk_rows > 64 : rows > 64)) return hipErrorInvalidValue;
  const long long total = (long long)rows * ld_dst;
  const int grid = (int)std::min<long long>((total + 255) / 256, 1024);
  if (dtype == DT_BF16)
    k_cvt_pad<uint16_t><<<grid, 256, 0, st>>>(src, rows, cols, (uint16_t*)dst, ld_dst, afrag, dst_f32,
                                              blk_rows, blk_elems);
  else
    k_cvt_pad<float><<<grid, 256, 0, st>>>(src, rows, cols, (float*)dst, ld_dst, afrag, dst_f32,
                                           blk_rows, blk_elems);
  return hipGetLastError();
}

template <typename T>
__global__ void k_bcast_row(const T* __restrict__ row, int cols, T* __restrict__ dst, int ld,
                            int rows) {
  const long long total = (long long)rows * cols;
  for (long long idx = blockIdx.x * (long long)blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % cols);
    const long long r = idx / cols;
    dst[r * ld + c] = row[c];
  }
}

hipError_t launch_bcast_row(int dtype, const void* row, int cols, void* dst, int ld_dst, int rows,
                            hipStream_t st) {
  const long long total = (long long)rows * cols;
  const int grid = (int)std::min<long long>((total + 255) / 256, 1024);
  if (dtype == DT_BF16)
    k_bcast_row<uint16_t><<<grid, 256, 0, st>>>((const uint16_t*)row, cols, (uint16_t*)dst, ld_dst, rows);
  else
    k_bcast_row<float><<<grid, 256, 0, st>>>((const float*)row, cols, (float*)dst, ld_dst, rows);
  return hipGetLastError();
}

}  // namespace vla
