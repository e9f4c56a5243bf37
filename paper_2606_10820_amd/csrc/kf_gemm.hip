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
  __device__ static inline void mma(const uint4& a, const uint4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};
template <>
struct Mfma<float> {
  __device__ static inline void mma(const uint4& a, const uint4& b, f32x4& c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
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
// the KV cache slot C + i of sequence b (the KV append of the step).
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
    T* dst;
    if (which == 0) {
      dst = Q + (size_t)m * d + c;
    } else {
      const int b = m / g.R, i = m - b * g.R;
      const int h = c / kg.dh, e = c - h * kg.dh;
      dst = kv + (size_t)b * kg.seq_stride() + kg.head_off(layer, which - 1, h) +
            (size_t)(st->C + i) * kg.dh + e;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[i] = from_f<T>(v[i] + bias[n + i]);
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
template <typename T, int BM, int BN, int WM, int WN, class Ep>
__global__ void __launch_bounds__(256)
    gemm_kernel(const T* __restrict__ A, int lda, const T* __restrict__ W, int ldw, int M, int N,
                int K, Ep ep) {
  constexpr int CH = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  constexpr int BK = 8 * CH;               // K per slab (128 bytes per row)
  constexpr int ROW = 9;                   // chunks per LDS row (8 + 1 padding)
  constexpr int MW = BM / WM, NW = BN / WN;
  constexpr int TM = MW / 16, TN = NW / 16;
  constexpr int LA = (BM * 8 + 255) / 256, LW = (BN * 8 + 255) / 256;
  static_assert(WM * WN == 4, "four wavefronts");
  static_assert(MW % 16 == 0 && NW % 16 == 0, "16x16 MFMA tiles");

  __shared__ uint4 sA[2][BM * ROW];
  __shared__ uint4 sW[2][BN * ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  uint4 ra[LA], rw[LW];
  const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);

  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      int c = tid + i * 256;
      int r = c >> 3, cc = c & 7;
      int gm = m0 + r;
      ra[i] = (c < BM * 8 && gm < M)
                  ? *reinterpret_cast<const uint4*>(A + (size_t)gm * lda + (size_t)kt * BK + cc * CH)
                  : z4;
    }
#pragma unroll
    for (int i = 0; i < LW; ++i) {
      int c = tid + i * 256;
      int r = c >> 3, cc = c & 7;
      int gn = n0 + r;
      rw[i] = (c < BN * 8 && gn < N)
                  ? *reinterpret_cast<const uint4*>(W + (size_t)gn * ldw + (size_t)kt * BK + cc * CH)
                  : z4;
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      int c = tid + i * 256;
      if (c < BM * 8) sA[buf][(c >> 3) * ROW + (c & 7)] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < LW; ++i) {
      int c = tid + i * 256;
      if (c < BN * 8) sW[buf][(c >> 3) * ROW + (c & 7)] = rw[i];
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      uint4 af[TN], bfr[TM];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
        af[tn] = sW[cur][(wn * NW + tn * 16 + (lane & 15)) * ROW + s * 4 + (lane >> 4)];
#pragma unroll
      for (int tm = 0; tm < TM; ++tm)
        bfr[tm] = sA[cur][(wm * MW + tm * 16 + (lane & 15)) * ROW + s * 4 + (lane >> 4)];
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) Mfma<T>::mma(af[tn], bfr[tm], acc[tn][tm]);
    }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

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
        ep.pval[(size_t)m * ep.n_tiles + blockIdx.x] = bv;
        ep.pidx[(size_t)m * ep.n_tiles + blockIdx.x] = bi;
      }
    }
  }
}

template <typename T, int BM, int BN, int WM, int WN, class Ep>
hipError_t run(const T* A, int lda, const T* W, int ldw, int M, int N, int K, const Ep& ep,
               hipStream_t s) {
  dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, Ep>), grid, dim3(256), 0, s, A, lda, W, ldw,
                     M, N, K, ep);
  return hipGetLastError();
}

// Tile choice by M (rows of activations).
template <typename T, class Ep>
hipError_t dispatch(const T* A, int lda, const T* W, int ldw, int M, int N, int K, const Ep& ep,
                    hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if (M <= 32) return run<T, 32, 64, 1, 4>(A, lda, W, ldw, M, N, K, ep, s);
  if (M <= 256) return run<T, 64, 64, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
  return run<T, 128, 128, 2, 2>(A, lda, W, ldw, M, N, K, ep, s);
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
  return run<T, 64, kHeadTileN, 2, 2>(A, K, W, K, M, Vpad, K, ep, s);
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
