// kf_gemm.hip -- MFMA GEMM family for the decode step on gfx950.
//
//   C[m][n] = epilogue( sum_k A[m][k] * W[n][k] ),   A: activations [M][K],
//   W: weights [N][K] (PyTorch Linear layout), fp32 accumulation.
//
// One workgroup of 4 wavefronts computes a BM x BN tile.  K is consumed in
// 128-byte slabs (64 bf16 / 32 fp32) staged through double-buffered LDS;
// each wavefront issues 16x16 MFMAs (v_mfma_f32_16x16x32_bf16 for bf16,
// v_mfma_f32_16x16x4_f32 for fp32) with the weight tile as the MFMA "A"
// operand and the activation tile as "B", so that each lane ends up holding
// four consecutive output columns of one row -- the natural unit for the
// vectorised epilogues.  Each lane feeds a 16-byte K-chunk of its row to the
// MFMA; both operands use the same chunk-to-k assignment, so the sum over k
// is exact whatever order the instruction uses inside a chunk.
#include <float.h>
#include <math.h>

#include "kf_internal.h"

namespace kf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte chunk

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(bf16 x) { return (float)x; }
template <typename T>
__device__ inline T from_f(float x);
template <>
__device__ inline float from_f<float>(float x) { return x; }
template <>
__device__ inline bf16 from_f<bf16>(float x) { return (bf16)x; }

// GELU, tanh form (GPT-2 style), evaluated with the device tanhf.
__device__ inline float gelu_f(float x) {
  const float c = 0.7978845608028654f;
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

template <typename T>
struct Mfma;
template <>
struct Mfma<bf16> {
  __device__ static inline void mma(const u32x4& a, const u32x4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <>
struct Mfma<float> {
  __device__ static inline void mma(const u32x4& a, const u32x4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0]), __uint_as_float(b[0]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1]), __uint_as_float(b[1]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[2]), __uint_as_float(b[2]), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[3]), __uint_as_float(b[3]), c, 0, 0, 0);
  }
};

// ------------------------------------------------------------ epilogues
// store4(m, n, v): v holds C[m][n .. n+3]; N is a multiple of 4.

template <typename T>
struct EpBias {
  T* out;
  int ldo;
  const float* bias;
  int gelu;
  __device__ inline void store4(int m, int n, f32x4 v) const {
    T* o = out + (size_t)m * ldo + n;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float x = v[i] + (bias ? bias[n + i] : 0.f);
      if (gelu) x = gelu_f(x);
      o[i] = from_f<T>(x);
    }
  }
};

struct EpResidual {
  float* X;
  int ldx;
  const float* bias;
  __device__ inline void store4(int m, int n, f32x4 v) const {
    float4* p = reinterpret_cast<float4*>(X + (size_t)m * ldx + n);
    float4 x = *p;
    x.x += v[0] + bias[n + 0];
    x.y += v[1] + bias[n + 1];
    x.z += v[2] + bias[n + 2];
    x.w += v[3] + bias[n + 3];
    *p = x;
  }
};

// QKV projection: q goes to Q [M][d]; k and v of row (b, i) go straight into
// the KV cache slot C + i of sequence b (the KV append of the step).  Keys are
// stored [slot][d_head] and values transposed, [d_head][slot], per head.
template <typename T>
struct EpQKV {
  T* Q;
  T* kv;
  const float* bias;
  const KfDevState* st;
  KfStepGeom g;
  KfKvGeom kg;
  int layer;
  __device__ inline void store4(int m, int n, f32x4 v) const {
    const int d = kg.H * kg.dh;
    const int which = n / d, c = n - which * d;
    if (which == 0) {
      T* dst = Q + (size_t)m * d + c;
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = from_f<T>(v[i] + bias[n + i]);
      return;
    }
    const int b = m / g.R, i = m - b * g.R;
    const int h = c / kg.dh, e = c - h * kg.dh;
    const int slot = st->C + i;
    T* base = kv + (size_t)b * kg.seq_stride() + kg.head_off(layer, which - 1, h);
    if (which == 1) {  // keys: [slot][dh]
      T* dst = base + (size_t)slot * kg.dh + e;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[r] = from_f<T>(v[r] + bias[n + r]);
    } else {           // values, transposed: [dh][slot]
#pragma unroll
      for (int r = 0; r < 4; ++r) base[(size_t)(e + r) * kg.T + slot] = from_f<T>(v[r] + bias[n + r]);
    }
  }
};

// Second noise-MLP layer: noise row m = (b, j) lands in residual row
// b*R + nr + j with its learned position C + nr + j added.
template <typename T>
struct EpNoiseOut {
  float* X;
  const float* bias;
  const T* pos;
  const KfDevState* st;
  KfStepGeom g;
  int d;
  __device__ inline void store4(int m, int n, f32x4 v) const {
    const int b = m / g.k, j = m - b * g.k;
    const int p = st->C + g.nr + j;
    float* x = X + ((size_t)b * g.R + g.nr + j) * d + n;
    const T* pe = pos + (size_t)p * d + n;
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = v[i] + bias[n + i] + to_f(pe[i]);
  }
};

// Head: no store; per-tile argmax partials (and optional fp32 logits).
struct EpHead {
  float* pval;
  int* pidx;
  float* logits;
  int V;
  int n_tiles;
};

template <typename Ep>
struct IsHead {
  static constexpr bool value = false;
};
template <>
struct IsHead<EpHead> {
  static constexpr bool value = true;
};

// ---------------------------------------------------------------- layout
// LDS tiles hold 8 16-byte chunks per row (one 128-byte K slab).  Chunk c of
// row r is stored at position c ^ ((r >> 1) & 7): sixteen lanes reading the
// same chunk of sixteen consecutive rows (one MFMA operand fetch) touch
// distinct 16-byte bank groups, and so do the 16-byte stores of a row.
constexpr int KCH = 8;
__device__ inline int swz(int r, int c) { return r * KCH + (c ^ ((r >> 1) & 7)); }

// Workgroups are dealt to the eight XCDs round-robin by linear id; give each
// XCD a contiguous run of tiles (M fastest) so that the workgroups sharing a
// weight strip share one L2.
__device__ inline int xcd_tile(int lin, int total) {
  const int q = total >> 3, r = total & 7;
  const int x = lin & 7, j = lin >> 3;
  return x * q + (x < r ? x : r) + j;
}

typedef const u32x4 __attribute__((address_space(1)))* gptr16;
__device__ inline u32x4 gload16(const void* p) { return *(gptr16)p; }

// Buffer resource over [base, base + bytes) and a 16-byte buffer load at a
// byte offset.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ inline u32x4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// ------------------------------------------------------------ A loaders
// An A loader stages one K slab of the BM-row activation tile.  Each thread
// owns L chunks of the slab: chunk c = tid + i*256 -> row c / 8, column chunk
// c % 8 (a row's chunks sit in 8 consecutive lanes).  Rows past the end
// re-read the last valid row: a tile row only feeds its own output row, which
// is never stored, so the loads need no predicate and stay branch-free.

// Plain: A is the compute-dtype matrix [M][lda].
template <typename T, int BM>
struct APlain {
  static constexpr int L = BM * KCH / 256;
  static constexpr int CH = 16 / (int)sizeof(T);
  static constexpr bool kNorm = false;
  static constexpr int kRegs = 4 * L;  // VGPRs per staged slab
  struct Stage {
    u32x4 r[L];
  };
  const T* A;
  int lda;
  int M;
  __device__ void init(int, int) {}
  __device__ void load(Stage& st, int m0, int k0, int tid) const {
#ifdef KF_GEMM_BUFLOAD
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(A, (uint32_t)((size_t)M * lda * sizeof(T)));
#endif
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int c = tid + i * 256, gr = m0 + c / KCH;
      const int rr = gr < M ? gr : M - 1;
#ifdef KF_GEMM_BUFLOAD
      st.r[i] = bload16(rs, (uint32_t)(((size_t)rr * lda + k0 + (c % KCH) * CH) * sizeof(T)));
#else
      st.r[i] = gload16(A + (size_t)rr * lda + k0 + (c % KCH) * CH);
#endif
    }
  }
  __device__ void store(const Stage& st, u32x4* __restrict__ lds, int tid) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int c = tid + i * 256;
      lds[swz(c / KCH, c % KCH)] = st.r[i];
    }
  }
  __device__ void finish(float2*, int, int) {}
  __device__ inline f32x4 apply(f32x4 acc, float2, int) const { return acc; }
};

// Which residual row feeds GEMM row m (MODE 0: row m; 1: noise row m of the
// step; 2: last real row of sequence m).
template <int MODE>
__device__ inline int map_row(int m, const KfStepGeom& g) {
  if constexpr (MODE == 1) return (m / g.k) * g.R + g.nr + (m % g.k);
  else if constexpr (MODE == 2) return m * g.R + g.nr - 1;
  else return m;
}

// LayerNorm folded into the GEMM.  For a row x (fp32 residual stream) with
// mean mu and rstd = 1 / sqrt(var + 1e-5), gain g and shift beta:
//   sum_k W[n][k] LN(x)_k = rstd * (sum_k W[n][k] g_k v_k - delta * c1[n]) + c2[n],
// with v = x - x_ref (x_ref = the row's first element: keeps the MFMA operand
// centred), delta = mu - x_ref, c1 = W g and c2 = W beta precomputed at weight
// load.  The operand staged in LDS is g * v in the compute dtype; the loader
// accumulates sum v and sum v^2 of its rows over the whole K loop (the
// workgroup sees every column of its rows), so no statistics pass is needed.
template <typename T, int BM, int MODE>
struct ANorm {
  static constexpr int L = BM * KCH / 256;
  static constexpr int CH = 16 / (int)sizeof(T);  // elements per staged chunk
  static constexpr int XW = CH / 4;               // 16-byte fp32 words per chunk
  static constexpr bool kNorm = true;
  static constexpr int kRegs = 4 * (L * XW + XW);
  struct Stage {
    u32x4 x[L][XW];
    u32x4 g[XW];
  };
  const float* X;
  int ldx;
  int M;
  const float* gain;
  const float* c1;
  const float* c2;
  KfStepGeom g;
  float xref[L], s1[L], s2[L];

  __device__ void init(int m0, int tid) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int gr = m0 + (tid + i * 256) / KCH;
      const int rr = gr < M ? gr : M - 1;
      xref[i] = X[(size_t)map_row<MODE>(rr, g) * ldx];
      s1[i] = 0.f;
      s2[i] = 0.f;
    }
  }
  __device__ void load(Stage& st, int m0, int k0, int tid) const {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int c = tid + i * 256, gr = m0 + c / KCH;
      const int rr = gr < M ? gr : M - 1;
      const float* p = X + (size_t)map_row<MODE>(rr, g) * ldx + k0 + (c % KCH) * CH;
#pragma unroll
      for (int w = 0; w < XW; ++w) st.x[i][w] = gload16(p + 4 * w);
    }
    const float* gp = gain + k0 + (tid % KCH) * CH;  // same column chunk for every i
#pragma unroll
    for (int w = 0; w < XW; ++w) st.g[w] = gload16(gp + 4 * w);
  }
  __device__ void store(const Stage& st, u32x4* __restrict__ lds, int tid) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int c = tid + i * 256;
      u32x4 out;
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int w = 0; w < XW; ++w)
#pragma unroll
          for (int e = 0; e < 4; e += 2) {
            const float v0 = __uint_as_float(st.x[i][w][e]) - xref[i];
            const float v1 = __uint_as_float(st.x[i][w][e + 1]) - xref[i];
            s1[i] += v0 + v1;
            s2[i] += v0 * v0 + v1 * v1;
            const bf16 b0 = (bf16)(v0 * __uint_as_float(st.g[w][e]));
            const bf16 b1 = (bf16)(v1 * __uint_as_float(st.g[w][e + 1]));
            out[w * 2 + e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, b0) |
                                 ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16);
          }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = __uint_as_float(st.x[i][0][e]) - xref[i];
          s1[i] += v;
          s2[i] += v * v;
          out[e] = __float_as_uint(v * __uint_as_float(st.g[0][e]));
        }
      }
      lds[swz(c / KCH, c % KCH)] = out;
    }
  }
  // Row statistics to LDS: stat[row] = (delta, rstd).
  __device__ void finish(float2* stat, int K, int tid) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      float a = s1[i], b = s2[i];
#pragma unroll
      for (int off = 1; off < KCH; off <<= 1) {
        a += __shfl_xor(a, off, 64);
        b += __shfl_xor(b, off, 64);
      }
      if ((tid % KCH) == 0) {
        const float delta = a / (float)K;
        const float var = fmaxf(b / (float)K - delta * delta, 0.f);
        stat[(tid + i * 256) / KCH] = make_float2(delta, 1.0f / sqrtf(var + 1e-5f));
      }
    }
  }
  __device__ inline f32x4 apply(f32x4 acc, float2 st, int n) const {
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = st.y * (acc[i] - st.x * c1[n + i]) + c2[n + i];
    return r;
  }
};

// One K slab of this wavefront's TN x TM block of 16x16 tiles.
template <typename T, int TM, int TN>
__device__ __forceinline__ void mma_slab(f32x4 (&acc)[TN][TM], const u32x4* __restrict__ la,
                                         const u32x4* __restrict__ lw, int arow, int wrow,
                                         int lane) {
#pragma unroll
  for (int s = 0; s < KCH / 4; ++s) {
    u32x4 af[TN], bfr[TM];
    const int ch = s * 4 + (lane >> 4);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) af[tn] = lw[swz(wrow + tn * 16, ch)];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) bfr[tm] = la[swz(arow + tm * 16, ch)];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) Mfma<T>::mma(af[tn], bfr[tm], acc[tn][tm]);
  }
}

template <int L, typename T>
__device__ __forceinline__ void gload_w(u32x4 (&r)[L], const T* __restrict__ base, int ld, int row0,
                                        int nrows, int k0, int tid) {
  constexpr int CH = 16 / (int)sizeof(T);
#ifdef KF_GEMM_BUFLOAD
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(base, (uint32_t)((size_t)nrows * ld * sizeof(T)));
#endif
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int c = tid + i * 256, gr = row0 + c / KCH;
    const int rr = gr < nrows ? gr : nrows - 1;
#ifdef KF_GEMM_BUFLOAD
    r[i] = bload16(rs, (uint32_t)(((size_t)rr * ld + k0 + (c % KCH) * CH) * sizeof(T)));
#else
    r[i] = gload16(base + (size_t)rr * ld + k0 + (c % KCH) * CH);
#endif
  }
}

template <int L>
__device__ __forceinline__ void sstore_w(const u32x4 (&r)[L], u32x4* __restrict__ lds, int tid) {
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int c = tid + i * 256;
    lds[swz(c / KCH, c % KCH)] = r[i];
  }
}

// ---------------------------------------------------------------- kernel
// Ring of S register stages over the K slabs (S divides the slab count): the
// prologue issues slabs 0..S-1; slab kt is stored to LDS buffer kt & 1 (last
// read by slab kt - 2, which every wavefront finished before the barrier of
// slab kt - 1), then its registers are refilled with slab kt + S, so S slabs
// are always in flight.  The last trip is peeled and issues no loads.
// Scheduling barriers keep each slab's loads in issue order, so the wait
// before a slab's LDS store covers only that slab.
template <typename T, int BM, int BN, int WM, int WN, int S, class AL, class Ep>
__global__ void __launch_bounds__(256)
    gemm_kernel(AL al, const T* __restrict__ W, int ldw, int M, int N, int K, Ep ep) {
  constexpr int CH = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  constexpr int BK = KCH * CH;             // K per slab
  constexpr int MW = BM / WM, NW = BN / WN;
  constexpr int TM = MW / 16, TN = NW / 16;
  constexpr int LW = BN * KCH / 256;
  static_assert(WM * WN == 4, "four wavefronts");
  static_assert(MW % 16 == 0 && NW % 16 == 0, "16x16 MFMA tiles");
  static_assert((BM * KCH) % 256 == 0 && (BN * KCH) % 256 == 0, "whole chunks per thread");
  static_assert(S % 2 == 0, "even ring depth (LDS buffer parity)");

  __shared__ u32x4 sA[2][BM * KCH];
  __shared__ u32x4 sW[2][BN * KCH];
  __shared__ float2 sStat[AL::kNorm ? BM : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int gm = (M + BM - 1) / BM, gn = (N + BN - 1) / BN;
  const int tile = xcd_tile(blockIdx.x, gm * gn);
  const int m0 = (tile % gm) * BM, n0 = (tile / gm) * BN;

  AL a = al;
  a.init(m0, tid);

  f32x4 acc[TN][TM];
#pragma unroll
  for (int x = 0; x < TN; ++x)
#pragma unroll
    for (int y = 0; y < TM; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int arow = wm * MW + (lane & 15), wrow = wn * NW + (lane & 15);
  const int trips = K / (BK * S);

  typename AL::Stage sa[S];
  u32x4 rw[S][LW];
#pragma unroll
  for (int i = 0; i < S; ++i) {
    a.load(sa[i], m0, i * BK, tid);
    gload_w<LW>(rw[i], W, ldw, n0, N, i * BK, tid);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int t = 0; t + 1 < trips; ++t) {
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int kn = (t * S + i + S) * BK;
      a.store(sa[i], sA[i & 1], tid);
      sstore_w<LW>(rw[i], sW[i & 1], tid);
      __syncthreads();
      a.load(sa[i], m0, kn, tid);
      gload_w<LW>(rw[i], W, ldw, n0, N, kn, tid);
      __builtin_amdgcn_sched_barrier(0);
      mma_slab<T, TM, TN>(acc, sA[i & 1], sW[i & 1], arow, wrow, lane);
    }
  }
#pragma unroll
  for (int i = 0; i < S; ++i) {
    a.store(sa[i], sA[i & 1], tid);
    sstore_w<LW>(rw[i], sW[i & 1], tid);
    __syncthreads();
    mma_slab<T, TM, TN>(acc, sA[i & 1], sW[i & 1], arow, wrow, lane);
  }
  if constexpr (AL::kNorm) {
    a.finish(sStat, K, tid);
    __syncthreads();
  }

  if constexpr (!IsHead<Ep>::value) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
        const int ml = wm * MW + tm * 16 + (lane & 15), m = m0 + ml;
        if (m < M && n < N) ep.store4(m, n, a.apply(acc[tn][tm], sStat[AL::kNorm ? ml : 0], n));
      }
  } else {
    // Row-wise argmax over this tile's columns: lane-local, then across the
    // four lane groups holding the same row, then across the WN wavefronts.
    __shared__ float redv[WN][BM];
    __shared__ int redi[WN][BM];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int mloc = wm * MW + tm * 16 + (lane & 15);
      const int m = m0 + mloc;
      const float2 st = sStat[AL::kNorm ? mloc : 0];
      float bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
        const f32x4 v = a.apply(acc[tn][tm], st, n);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (n + i < ep.V && v[i] > bv) { bv = v[i]; bi = n + i; }
        if (ep.logits && m < M) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n + i < ep.V) ep.logits[(size_t)m * ep.V + n + i] = v[i];
        }
      }
#pragma unroll
      for (int off = 16; off < 64; off <<= 1) {
        float ov = __shfl_xor(bv, off, 64);
        int oi = __shfl_xor(bi, off, 64);
        if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
      }
      if ((lane >> 4) == 0) {
        redv[wn][mloc] = bv;
        redi[wn][mloc] = bi;
      }
    }
    __syncthreads();
    if (tid < BM) {
      float bv = redv[0][tid];
      int bi = redi[0][tid];
#pragma unroll
      for (int w = 1; w < WN; ++w) {
        float ov = redv[w][tid];
        int oi = redi[w][tid];
        if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
      }
      const int m = m0 + tid;
      if (m < M) {
        const int nt = n0 / BN;
        ep.pval[(size_t)m * ep.n_tiles + nt] = bv;
        ep.pidx[(size_t)m * ep.n_tiles + nt] = bi;
      }
    }
  }
}

// Ring depth: the deepest of {12, 6, 2} that divides the slab count and keeps
// the staged slabs within 192 registers per thread (deeper rings are not even
// instantiated for tiles whose stages would not fit).
template <typename T, int BM, int BN, int WM, int WN, class AL, class Ep>
hipError_t launch_gemm(const AL& al, const T* W, int ldw, int M, int N, int K, const Ep& ep,
                       hipStream_t s) {
  constexpr int BK = KCH * 16 / (int)sizeof(T);
  constexpr int LW = BN * KCH / 256;
  constexpr int per = AL::kRegs + 4 * LW;
  const int tiles = ((N + BN - 1) / BN) * ((M + BM - 1) / BM);
  const int nk = K / BK;
  if constexpr (12 * per <= 192) {
    if (nk % 12 == 0) {
      hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, 12, AL, Ep>), dim3(tiles), dim3(256), 0,
                         s, al, W, ldw, M, N, K, ep);
      return hipGetLastError();
    }
  }
  if constexpr (6 * per <= 192) {
    if (nk % 6 == 0) {
      hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, 6, AL, Ep>), dim3(tiles), dim3(256), 0, s,
                         al, W, ldw, M, N, K, ep);
      return hipGetLastError();
    }
  }
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, 2, AL, Ep>), dim3(tiles), dim3(256), 0, s, al,
                     W, ldw, M, N, K, ep);
  return hipGetLastError();
}

// Loader arguments independent of the tile shape; launch() instantiates the
// loader for the chosen tile.
template <typename T>
struct PlainArgs {
  const T* A;
  int lda, M;
  template <int BM, int BN, int WM, int WN, class Ep>
  hipError_t launch(const T* W, int ldw, int Mr, int N, int K, const Ep& ep, hipStream_t s) const {
    APlain<T, BM> al;
    al.A = A;
    al.lda = lda;
    al.M = M;
    return launch_gemm<T, BM, BN, WM, WN>(al, W, ldw, Mr, N, K, ep, s);
  }
};

template <typename T, int MODE>
struct NormArgs {
  const float* X;
  int ldx, M;
  const float* gain;
  const float* c1;
  const float* c2;
  KfStepGeom g;
  template <int BM, int BN, int WM, int WN, class Ep>
  hipError_t launch(const T* W, int ldw, int Mr, int N, int K, const Ep& ep, hipStream_t s) const {
    ANorm<T, BM, MODE> al;
    al.X = X;
    al.ldx = ldx;
    al.M = M;
    al.gain = gain;
    al.c1 = c1;
    al.c2 = c2;
    al.g = g;
    return launch_gemm<T, BM, BN, WM, WN>(al, W, ldw, Mr, N, K, ep, s);
  }
};

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Tile choice: the largest tile that still gives at least one workgroup per
// CU (256), else the smallest tile.
template <typename T, class ALP, class Ep>
hipError_t dispatch(const ALP& alp, const T* W, int ldw, int M, int N, int K, const Ep& ep,
                    hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  constexpr int kFill = 256;
  if (cdiv(M, 128) * cdiv(N, 128) >= kFill)
    return alp.template launch<128, 128, 2, 2>(W, ldw, M, N, K, ep, s);
  if (cdiv(M, 64) * cdiv(N, 128) >= kFill)
    return alp.template launch<64, 128, 2, 2>(W, ldw, M, N, K, ep, s);
  if (cdiv(M, 64) * cdiv(N, 64) >= kFill)
    return alp.template launch<64, 64, 2, 2>(W, ldw, M, N, K, ep, s);
  if (cdiv(M, 32) * cdiv(N, 64) >= kFill)
    return alp.template launch<32, 64, 2, 2>(W, ldw, M, N, K, ep, s);
  return alp.template launch<32, 32, 2, 2>(W, ldw, M, N, K, ep, s);
}

// c1[n] = sum_k W[n][k] g[k], c2[n] = sum_k W[n][k] beta[k]: one wavefront per
// output column, fixed summation order.
template <typename T>
__global__ void __launch_bounds__(256)
    ln_fold_kernel(const T* __restrict__ W, const float* __restrict__ g,
                   const float* __restrict__ beta, int N, int K, float* c1, float* c2) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (n >= N) return;
  float a = 0.f, b = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float w = to_f(W[(size_t)n * K + k]);
    a += w * g[k];
    b += w * beta[k];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_xor(a, off, 64);
    b += __shfl_xor(b, off, 64);
  }
  if (lane == 0) {
    c1[n] = a;
    c2[n] = b;
  }
}

}  // namespace

template <typename T>
hipError_t gemm_bias(const T* A, const T* W, int M, int N, int K, const float* bias, Act act,
                     T* out, int ldo, hipStream_t s) {
  EpBias<T> ep{out, ldo, bias, act == Act::Gelu ? 1 : 0};
  return dispatch<T>(PlainArgs<T>{A, K, M}, W, K, M, N, K, ep, s);
}

template <typename T>
hipError_t gemm_residual(const T* A, const T* W, int M, int N, int K, const float* bias, float* X,
                         hipStream_t s) {
  EpResidual ep{X, N, bias};
  return dispatch<T>(PlainArgs<T>{A, K, M}, W, K, M, N, K, ep, s);
}

template <typename T>
hipError_t gemm_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                          const T* pos, float* X, KfStepGeom g, const KfDevState* st,
                          hipStream_t s) {
  EpNoiseOut<T> ep{X, bias, pos, st, g, d};
  return dispatch<T>(PlainArgs<T>{A, K, M}, W, K, M, d, K, ep, s);
}

template <typename T>
hipError_t gemm_qkv_ln(const float* X, const LnFold& ln, const T* W, int M, int d,
                       const float* bias, T* Q, T* kv, KfStepGeom g, KfKvGeom kg, int layer,
                       const KfDevState* st, hipStream_t s) {
  EpQKV<T> ep{Q, kv, bias, st, g, kg, layer};
  NormArgs<T, 0> na{X, d, M, ln.gain, ln.c1, ln.c2, g};
  return dispatch<T>(na, W, d, M, 3 * d, d, ep, s);
}

template <typename T>
hipError_t gemm_up_ln(const float* X, const LnFold& ln, const T* W, int M, int N, int d,
                      const float* bias, T* out, hipStream_t s) {
  EpBias<T> ep{out, N, bias, 1};
  NormArgs<T, 0> na{X, d, M, ln.gain, ln.c1, ln.c2, KfStepGeom{}};
  return dispatch<T>(na, W, d, M, N, d, ep, s);
}

template <typename T>
hipError_t gemm_head_ln(const float* X, const LnFold& ln, const T* W, int M, int Vpad, int V,
                        int d, int gather, KfStepGeom g, float* pval, int* pidx, float* logits,
                        hipStream_t s) {
  if (M <= 0) return hipSuccess;
  EpHead ep{pval, pidx, logits, V, Vpad / kHeadTileN};
  auto go = [&](auto na) {
    if (M <= 32) return na.template launch<32, kHeadTileN, 1, 4>(W, d, M, Vpad, d, ep, s);
    if (M <= 512) return na.template launch<64, kHeadTileN, 2, 2>(W, d, M, Vpad, d, ep, s);
    return na.template launch<128, kHeadTileN, 2, 2>(W, d, M, Vpad, d, ep, s);
  };
  if (gather == 2) return go(NormArgs<T, 2>{X, d, M, ln.gain, ln.c1, ln.c2, g});
  return go(NormArgs<T, 1>{X, d, M, ln.gain, ln.c1, ln.c2, g});
}

template <typename T>
hipError_t launch_ln_fold(const T* W, const float* g, const float* beta, int N, int K, float* c1,
                          float* c2, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  hipLaunchKernelGGL(ln_fold_kernel<T>, dim3((N + 3) / 4), dim3(256), 0, s, W, g, beta, N, K, c1,
                     c2);
  return hipGetLastError();
}

#define KF_INST(T)                                                                                 \
  template hipError_t gemm_bias<T>(const T*, const T*, int, int, int, const float*, Act, T*, int, \
                                   hipStream_t);                                                   \
  template hipError_t gemm_residual<T>(const T*, const T*, int, int, int, const float*, float*,   \
                                       hipStream_t);                                               \
  template hipError_t gemm_noise_out<T>(const T*, const T*, int, int, int, const float*,          \
                                        const T*, float*, KfStepGeom, const KfDevState*,           \
                                        hipStream_t);                                              \
  template hipError_t gemm_qkv_ln<T>(const float*, const LnFold&, const T*, int, int,             \
                                     const float*, T*, T*, KfStepGeom, KfKvGeom, int,              \
                                     const KfDevState*, hipStream_t);                              \
  template hipError_t gemm_up_ln<T>(const float*, const LnFold&, const T*, int, int, int,         \
                                    const float*, T*, hipStream_t);                                \
  template hipError_t gemm_head_ln<T>(const float*, const LnFold&, const T*, int, int, int, int,  \
                                      int, KfStepGeom, float*, int*, float*, hipStream_t);         \
  template hipError_t launch_ln_fold<T>(const T*, const float*, const float*, int, int, float*,   \
                                        float*, hipStream_t);
KF_INST(float)
KF_INST(bf16)
#undef KF_INST

}  // namespace kf
