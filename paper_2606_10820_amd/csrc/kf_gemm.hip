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

// ---------------------------------------------------------------- kernel
// LDS tiles hold KCH 16-byte chunks per row (one K slab of KCH * 16 bytes).
// Chunk c of row r is stored at position c ^ f(r) with f(r) = (r >> 1) & 7 for
// 8 chunks (128-byte rows) and r & 15 for 16 chunks (256-byte rows): sixteen
// lanes reading the same chunk of sixteen consecutive rows (one MFMA operand
// fetch) then touch sixteen distinct 16-byte bank groups, and so do the
// 16-byte stores of a row.
template <int KCH>
__device__ inline int swz(int r, int c) {
  if constexpr (KCH == 8) return r * 8 + (c ^ ((r >> 1) & 7));
  else return r * KCH + (c ^ (r & (KCH - 1)));
}

// Workgroups are dealt to the eight XCDs round-robin by linear id; give each
// XCD a contiguous run of tiles (M fastest) so that the workgroups sharing a
// weight strip share one L2.
__device__ inline int xcd_tile(int lin, int total) {
  const int q = total >> 3, r = total & 7;
  const int x = lin & 7, j = lin >> 3;
  return x * q + (x < r ? x : r) + j;
}

typedef const u32x4 __attribute__((address_space(1)))* gptr16;

// Load this thread's chunks of one K slab (KCH chunks per row) of a tile
// starting at global row row0.  Rows past the end re-read the last valid row:
// a tile row only ever feeds its own output row or column, and those outputs
// are never stored, so the loads need no predicate (and stay branch-free).
template <int L, int KCH, typename T>
__device__ __forceinline__ void gload_tile(u32x4 (&r)[L], const T* __restrict__ base, int ld,
                                           int row0, int nrows, int k0, int tid) {
  constexpr int CH = 16 / (int)sizeof(T);
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int c = tid + i * 256, gr = row0 + c / KCH;
    const int rr = gr < nrows ? gr : nrows - 1;
    r[i] = *(gptr16)(const void*)(base + (size_t)rr * ld + k0 + (c % KCH) * CH);
  }
}

template <int L, int KCH>
__device__ __forceinline__ void sstore_tile(const u32x4 (&r)[L], u32x4* __restrict__ lds, int tid) {
#pragma unroll
  for (int i = 0; i < L; ++i) {
    const int c = tid + i * 256;
    lds[swz<KCH>(c / KCH, c % KCH)] = r[i];
  }
}

// One K slab of this wavefront's TN x TM block of 16x16 tiles.
template <typename T, int TM, int TN, int KCH>
__device__ __forceinline__ void mma_slab(f32x4 (&acc)[TN][TM], const u32x4* __restrict__ la,
                                         const u32x4* __restrict__ lw, int arow, int wrow,
                                         int lane) {
#pragma unroll
  for (int s = 0; s < KCH / 4; ++s) {
    u32x4 af[TN], bfr[TM];
    const int ch = s * 4 + (lane >> 4);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) af[tn] = lw[swz<KCH>(wrow + tn * 16, ch)];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) bfr[tm] = la[swz<KCH>(arow + tm * 16, ch)];
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) Mfma<T>::mma(af[tn], bfr[tm], acc[tn][tm]);
  }
}

template <typename T, int BM, int BN, int WM, int WN, int KCH, class Ep>
__global__ void __launch_bounds__(256)
    gemm_kernel(const T* __restrict__ A, int lda, const T* __restrict__ W, int ldw, int M, int N,
                int K, Ep ep) {
  constexpr int CH = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  constexpr int BK = KCH * CH;             // K per slab (KCH * 16 bytes per row)
  constexpr int MW = BM / WM, NW = BN / WN;
  constexpr int TM = MW / 16, TN = NW / 16;
  constexpr int LA = BM * KCH / 256, LW = BN * KCH / 256;
  static_assert(WM * WN == 4, "four wavefronts");
  static_assert(MW % 16 == 0 && NW % 16 == 0, "16x16 MFMA tiles");
  static_assert((BM * KCH) % 256 == 0 && (BN * KCH) % 256 == 0, "whole chunks per thread");

  __shared__ u32x4 sA[2][BM * KCH];
  __shared__ u32x4 sW[2][BN * KCH];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int gm = (M + BM - 1) / BM, gn = (N + BN - 1) / BN;
  const int tile = xcd_tile(blockIdx.x, gm * gn);
  const int m0 = (tile % gm) * BM, n0 = (tile / gm) * BN;

  // two register stages of prefetched chunks (loads run two slabs ahead)
  u32x4 ra0[LA], rw0[LW], ra1[LA], rw1[LW];

  f32x4 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int arow = wm * MW + (lane & 15), wrow = wn * NW + (lane & 15);
  const int nk = K / BK;
  // Prefetches are issued unconditionally (past the last slab they re-read
  // it) so that the count of loads in flight is the same on every path and
  // the waits before each LDS store cover only the older slab.
  auto kofs = [nk](int k) { return (k < nk ? k : nk - 1) * BK; };
  gload_tile<LA, KCH>(ra0, A, lda, m0, M, 0, tid);
  gload_tile<LW, KCH>(rw0, W, ldw, n0, N, 0, tid);
  gload_tile<LA, KCH>(ra1, A, lda, m0, M, kofs(1), tid);
  gload_tile<LW, KCH>(rw1, W, ldw, n0, N, kofs(1), tid);
  sstore_tile<LA, KCH>(ra0, sA[0], tid);
  sstore_tile<LW, KCH>(rw0, sW[0], tid);
  __syncthreads();
  // Slab kt is in LDS buffer kt&1; register stage kt&1 is free, stage
  // (kt+1)&1 holds slab kt+1.  Pairs of slabs per trip keep the register
  // stages statically addressed; an odd last slab is peeled.
  int kt = 0;
  for (; kt + 2 <= nk; kt += 2) {
    gload_tile<LA, KCH>(ra0, A, lda, m0, M, kofs(kt + 2), tid);
    gload_tile<LW, KCH>(rw0, W, ldw, n0, N, kofs(kt + 2), tid);
    mma_slab<T, TM, TN, KCH>(acc, sA[0], sW[0], arow, wrow, lane);
    sstore_tile<LA, KCH>(ra1, sA[1], tid);
    sstore_tile<LW, KCH>(rw1, sW[1], tid);
    __syncthreads();
    gload_tile<LA, KCH>(ra1, A, lda, m0, M, kofs(kt + 3), tid);
    gload_tile<LW, KCH>(rw1, W, ldw, n0, N, kofs(kt + 3), tid);
    mma_slab<T, TM, TN, KCH>(acc, sA[1], sW[1], arow, wrow, lane);
    // unconditional: past the end it rewrites buffer 0, which nothing reads
    // any more (an odd last slab has kt + 2 == nk - 1 and is the real one)
    sstore_tile<LA, KCH>(ra0, sA[0], tid);
    sstore_tile<LW, KCH>(rw0, sW[0], tid);
    __syncthreads();
  }
  if (kt < nk) mma_slab<T, TM, TN, KCH>(acc, sA[0], sW[0], arow, wrow, lane);

  if constexpr (!IsHead<Ep>::value) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
        const int m = m0 + wm * MW + tm * 16 + (lane & 15);
        if (m < M && n < N) ep.store4(m, n, acc[tn][tm]);
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
      float bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = acc[tn][tm][i];
          if (n + i < ep.V && v > bv) { bv = v; bi = n + i; }
        }
        if (ep.logits && m < M) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (n + i < ep.V) ep.logits[(size_t)m * ep.V + n + i] = acc[tn][tm][i];
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

template <typename T, int BM, int BN, int WM, int WN, int KCH = 8, class Ep>
hipError_t run(const T* A, int lda, const T* W, int ldw, int M, int N, int K, const Ep& ep,
               hipStream_t s) {
  const int tiles = ((N + BN - 1) / BN) * ((M + BM - 1) / BM);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, KCH, Ep>), dim3(tiles), dim3(256), 0, s, A,
                     lda, W, ldw, M, N, K, ep);
  return hipGetLastError();
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Tile choice: the largest tile that still gives at least one workgroup per
// CU (256), else the smallest tile.
template <typename T, class Ep>
hipError_t dispatch(const T* A, int lda, const T* W, int ldw, int M, int N, int K, const Ep& ep,
                    hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  constexpr int kFill = 256;
  if (cdiv(M, 128) * cdiv(N, 128) >= kFill) return run<T, 128, 128, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
  if (cdiv(M, 64) * cdiv(N, 128) >= kFill) return run<T, 64, 128, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
  if (cdiv(M, 64) * cdiv(N, 64) >= kFill) return run<T, 64, 64, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
  if (cdiv(M, 32) * cdiv(N, 64) >= kFill) return run<T, 32, 64, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
  return run<T, 32, 32, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
}

}  // namespace

template <typename T>
hipError_t gemm_bias(const T* A, const T* W, int M, int N, int K, const float* bias, Act act,
                     T* out, int ldo, hipStream_t s) {
  EpBias<T> ep{out, ldo, bias, act == Act::Gelu ? 1 : 0};
  return dispatch<T>(A, K, W, K, M, N, K, ep, s);
}

template <typename T>
hipError_t gemm_residual(const T* A, const T* W, int M, int N, int K, const float* bias, float* X,
                         hipStream_t s) {
  EpResidual ep{X, N, bias};
  return dispatch<T>(A, K, W, K, M, N, K, ep, s);
}

template <typename T>
hipError_t gemm_qkv(const T* A, const T* W, int M, int d, const float* bias, T* Q, T* kv,
                    KfStepGeom g, KfKvGeom kg, int layer, const KfDevState* st, hipStream_t s) {
  EpQKV<T> ep{Q, kv, bias, st, g, kg, layer};
  return dispatch<T>(A, d, W, d, M, 3 * d, d, ep, s);
}

template <typename T>
hipError_t gemm_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                          const T* pos, float* X, KfStepGeom g, const KfDevState* st,
                          hipStream_t s) {
  EpNoiseOut<T> ep{X, bias, pos, st, g, d};
  return dispatch<T>(A, K, W, K, M, d, K, ep, s);
}

template <typename T>
hipError_t gemm_head(const T* A, const T* W, int M, int Vpad, int V, int K, float* pval,
                     int* pidx, float* logits, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  EpHead ep{pval, pidx, logits, V, Vpad / kHeadTileN};
  if (M <= 32) return run<T, 32, kHeadTileN, 1, 4>(A, K, W, K, M, Vpad, K, ep, s);
  if (M <= 512) return run<T, 64, kHeadTileN, 2, 2>(A, K, W, K, M, Vpad, K, ep, s);
  return run<T, 128, kHeadTileN, 2, 2>(A, K, W, K, M, Vpad, K, ep, s);
}

#define KF_INST(T)                                                                                 \
  template hipError_t gemm_bias<T>(const T*, const T*, int, int, int, const float*, Act, T*, int, \
                                   hipStream_t);                                                   \
  template hipError_t gemm_residual<T>(const T*, const T*, int, int, int, const float*, float*,   \
                                       hipStream_t);                                               \
  template hipError_t gemm_qkv<T>(const T*, const T*, int, int, const float*, T*, T*, KfStepGeom, \
                                  KfKvGeom, int, const KfDevState*, hipStream_t);                  \
  template hipError_t gemm_noise_out<T>(const T*, const T*, int, int, int, const float*,          \
                                        const T*, float*, KfStepGeom, const KfDevState*,           \
                                        hipStream_t);                                              \
  template hipError_t gemm_head<T>(const T*, const T*, int, int, int, int, float*, int*, float*,  \
                                   hipStream_t);
KF_INST(float)
KF_INST(bf16)
#undef KF_INST

}  // namespace kf
