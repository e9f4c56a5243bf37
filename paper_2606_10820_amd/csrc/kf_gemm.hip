// kf_gemm.hip -- MFMA GEMM family for the decode step on gfx950.
//
//   C[m][n] = epilogue( sum_k A[m][k] * W[n][k] ),   A: activations [M][K],
//   W: weights [N][K] (PyTorch Linear layout), fp32 accumulation.
//
// One workgroup of 4 or 8 wavefronts computes a BM x BN tile.  K is consumed in
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

#include <type_traits>

#include "kf_internal.h"
#include "kf_lds.h"

namespace kf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(bf16 x) { return (float)x; }
template <typename T>
__device__ inline T from_f(float x);
template <>
__device__ inline float from_f<float>(float x) { return x; }
template <>
__device__ inline bf16 from_f<bf16>(float x) { return (bf16)x; }

// GELU, tanh form (GPT-2 style): 0.5 x (1 + tanh u) with u = c (x + 0.044715 x^3),
// evaluated as x * sigmoid(2u) = x / (1 + exp(-2u)), the same function.  The
// exponential is 2^z with z = -2u log2(e) = x (k0 + k1 x^2) (log2(e) folded into
// the constants), and the quotient is x times the hardware reciprocal (about
// 1 ulp): a full-precision division would cost ten instructions per element,
// and the epilogue of a large GEMM is bound by this arithmetic.  Saturates
// correctly at both ends: 2^z -> inf gives -0, 2^z -> 0 gives x.
__device__ inline float gelu_f(float x) {
  constexpr float k0 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
  constexpr float k1 = 0.044715f * k0;
  const float z = x * fmaf(k1, x * x, k0);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

// n / d for n >= 0 and a wave-uniform d > 0: a shift when d is a power of two
// (head widths, rows per sequence at k = 1, 2, 4), else the integer division.
__device__ inline int div_u(int n, int d) {
  return (d & (d - 1)) == 0 ? n >> __builtin_ctz((unsigned)d) : n / d;
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
// store8(m, n, v): v holds C[m][n .. n+7] with the bias (and a folded
// LayerNorm) already applied; n is a multiple of 8.  The kernel stages each
// tile through LDS so that consecutive lanes store consecutive 8-column chunks
// of a row.  Epilogues that write the residual stream (kStats) leave in v the
// eight values written and name their stream row (srow); the kernel then
// writes the LayerNorm partial sums of every 16-column group of that row to
// lnst [rows][cols() / 16] as (sum x, sum x^2), which the next
// LayerNorm-folded GEMM reads instead of recomputing row statistics.
// Eight consecutive values to T memory (16-byte aligned for bf16: one store).
template <typename T>
__device__ inline void put8(T* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[2 * i]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[2 * i + 1]) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  } else {
    reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// put8 for the KV append: a nontemporal store (the cache is streamed, not
// reused from the caches; see the decode attention's loads).
typedef unsigned int u32x4s_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2s_t __attribute__((ext_vector_type(2)));
template <typename T>
__device__ inline void put8_stream(T* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    u32x4s_t w;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[2 * i]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[2 * i + 1]) << 16);
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4s_t*>(p));
  } else {
    put8(p, v);
  }
}

template <typename T>
__device__ inline void get8(const T* p, float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    const uint4 q = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
    const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

template <typename T>
struct EpBias {
  T* out;
  int ldo;
  const float* bias;
  int gelu;
  static constexpr bool kStats = false;
  __device__ inline void store8(int m, int n, float (&v)[8]) const {
    if (gelu) {
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = gelu_f(v[i]);
    }
    put8(out + (size_t)m * ldo + n, v);
  }
};

// Residual update X += C + bias.  With a 16-bit compute dtype the updated row
// is also written to Xh, the compute-dtype copy of the residual stream that the
// LayerNorm-folded GEMMs read (for fp32, Xh is X itself).
template <typename T, bool ROWS = false>
struct EpResidual {
  float* X;
  T* Xh;
  int ldx;
  const float* bias;
  float2* lnst;
  // With ROWS the GEMM covers rk rows per sequence out of rR: GEMM row m is
  // stream row (m / rk) rR + rnr + m % rk (the head rows of a step).
  int rk = 0, rR = 0, rnr = 0;
  static constexpr bool kStats = true;
  __device__ inline int srow(int m) const {
    if constexpr (ROWS) {
      const int b = div_u(m, rk);
      return b * rR + rnr + (m - b * rk);
    } else {
      return m;
    }
  }
  __device__ inline int cols() const { return ldx; }
  __device__ inline void store8(int m, int n, float (&v)[8]) const {
    float x[8];
    pre8(m, n, x);
    store8_pre(m, n, v, x);
  }
  // The same in two halves, for kernels that load the old values early.
  __device__ inline void pre8(int m, int n, float (&x)[8]) const {
    get8(X + (size_t)srow(m) * ldx + n, x);
  }
  __device__ inline void store8_pre(int m, int n, float (&v)[8], const float (&x)[8]) const {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += x[i];
    const size_t r = (size_t)srow(m);
    put8(X + r * ldx + n, v);
    if constexpr (sizeof(T) == 2) put8(Xh + r * ldx + n, v);
  }
};
template <class Ep>
struct HasPre : std::false_type {};
template <typename T, bool ROWS>
struct HasPre<EpResidual<T, ROWS>> : std::true_type {};

// QKV projection: q goes to Q [M][d]; k and v of row (b, i) go straight into
// cache slot C_b + i of sequence b (the KV append of the step), in the page
// that holds it: keys [slot][d_head] and values transposed, [d_head][slot], per
// head.  An 8-column chunk never straddles q/k/v or two heads (d_head >= 32).
// Rotary positions (RoFormer) on 8 consecutive columns e..e+7 of one head
// (e even): pairs (e + 2r, e + 2r + 1) with pair index i = e/2 + r < d_rot/2
// turn by the table angle of position p (cs [n_ctx][d_rot/2] = cos, sin).
__device__ inline void rotate8(float (&v)[8], const float2* cs, int dr, int p, int e) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = e / 2 + r;
    if (2 * i < dr) {
      const float2 t = cs[(size_t)p * (dr / 2) + i];
      const float x0 = v[2 * r], x1 = v[2 * r + 1];
      v[2 * r] = x0 * t.x - x1 * t.y;
      v[2 * r + 1] = x0 * t.y + x1 * t.x;
    }
  }
}

// A run of len <= 4 consecutive elements starting at p, whose element 0 sits
// a elements into an aligned group of 4: the widest aligned stores.
template <typename T>
__device__ inline void put_run4(T* p, int a, const float* v, int len) {
  static_assert(kVBlk == 4, "runs of one value block");
  if constexpr (sizeof(T) == 2) {
    auto pair = [&](int j) {
      return (uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[j]) |
             ((uint32_t)__builtin_bit_cast(uint16_t, (bf16)v[j + 1]) << 16);
    };
    if (len == 4) {  // a == 0: one 8-byte store, nontemporal (see put8_stream)
      const u32x2s_t w = {pair(0), pair(2)};
      __builtin_nontemporal_store(w, reinterpret_cast<u32x2s_t*>(p));
      return;
    }
    for (int j = 0; j < len;) {
      if (((a + j) & 1) == 0 && j + 1 < len) {
        *reinterpret_cast<uint32_t*>(p + j) = pair(j);
        j += 2;
      } else {
        p[j] = (bf16)v[j];
        ++j;
      }
    }
  } else {
    if (len == 4) {
      *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
      return;
    }
    for (int j = 0; j < len; ++j) p[j] = v[j];
  }
}

template <typename T>
struct EpQKV {
  T* Q;
  T* kv;
  const float* bias;
  const KfDevState* st;
  KfStepGeom g;
  KfKvGeom kg;
  int layer;
  const float2* rope;  // rotary table, or null
  static constexpr bool kStats = false;
  __device__ inline void store8(int m, int n, float (&v)[8]) const {
    const int d = kg.H * kg.dh;
    const int which = (n >= d) + (n >= 2 * d), c = n - which * d;  // n < 3d
    if (which == 0 && !rope) {
      put8(Q + (size_t)m * d + c, v);
      return;
    }
    const int b = div_u(m, g.R), i = m - b * g.R;
    const int slot = g.ctx(st, b) + i;  // this row's position and cache slot
    const int h = div_u(c, kg.dh), e = c - h * kg.dh;
    if (rope && which < 2) rotate8(v, rope, kg.dh < 64 ? kg.dh : 64, slot, e);
    if (which == 0) {
      put8(Q + (size_t)m * d + c, v);
      return;
    }
    const int r0 = (unsigned)slot % kPage;
    T* base = kv + kg.page_base(g.slot(b), slot) + kg.head_off(layer, which - 1, h);
    if (which == 1) {  // keys: [slot][dh]
      put8_stream(base + (size_t)r0 * kg.dh + e, v);
    } else {           // values, transposed in 8-slot blocks
#pragma unroll
      for (int r = 0; r < 8; ++r) base[KfKvGeom::vt_off(slot, e + r, kg.dh)] = from_f<T>(v[r]);
    }
  }
  // Value tiles (column_tile) are stored by column: v holds rows m..m+7 (those
  // < M) of value column n.  Rows that are consecutive slots of one sequence
  // within one value block are one contiguous run, and consecutive lanes hold
  // consecutive value rows, whose runs are adjacent.
  __device__ inline bool column_tile(int n0) const { return n0 >= 2 * kg.H * kg.dh; }
  //
  // Every index into v is a compile-time constant (a run-time index would put
  // v in scratch memory): each group of 4 rows is one aligned 4-slot block of
  // one sequence (one 8-byte store) in the common case, else it is written as
  // aligned pairs of slots and single slots.
  __device__ inline T* vslot(int mr, int e, unsigned ho, int& i, int& slot) const {
    const int b = div_u(mr, g.R);
    i = mr - b * g.R;
    slot = g.ctx(st, b) + i;
    return kv + kg.page_base(g.slot(b), slot) + ho + KfKvGeom::vt_off(slot, e, kg.dh);
  }
  __device__ inline void store_col8(int m, int n, const float (&v)[8], int M) const {
    const int c = n - 2 * kg.H * kg.dh, h = div_u(c, kg.dh), e = c - h * kg.dh;
    const unsigned ho = kg.head_off(layer, 1, h);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int mq = m + 4 * q;
      if (mq >= M) break;
      int i, slot;
      T* p = vslot(mq, e, ho, i, slot);
      if ((slot & 3) == 0 && i + 4 <= g.R && mq + 4 <= M) {
        put_run4(p, 0, &v[4 * q], 4);
        continue;
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {  // rows mq + 2t, mq + 2t + 1
        const int mt = mq + 2 * t;
        if (mt >= M) break;
        int it, st0;
        T* pt = vslot(mt, e, ho, it, st0);
        if ((st0 & 1) == 0 && it + 2 <= g.R && mt + 2 <= M) {
          put_run4(pt, 0, &v[4 * q + 2 * t], 2);
          continue;
        }
        *pt = from_f<T>(v[4 * q + 2 * t]);
        if (mt + 1 < M) {
          T* p1 = vslot(mt + 1, e, ho, it, st0);
          *p1 = from_f<T>(v[4 * q + 2 * t + 1]);
        }
      }
    }
  }
};
template <typename Ep>
struct HasColumns {
  static constexpr bool value = false;
};
template <typename T>
struct HasColumns<EpQKV<T>> {
  static constexpr bool value = true;
};

// Second noise-MLP layer: noise row m = (b, j) lands in residual row
// b*R + nr + j with its learned position C_b + nr + j added, and, for a
// temperature-conditioned model, the temperature embedding of b's slot.
template <typename T>
struct EpNoiseOut {
  float* X;
  T* Xh;
  const float* bias;
  const T* pos;
  const T* temb;  // per-slot temperature embedding [slots][d], or null
  const KfDevState* st;
  KfStepGeom g;
  int d;
  float2* lnst;
  static constexpr bool kStats = true;
  __device__ inline int cols() const { return d; }
  __device__ inline int srow(int m) const {
    const int b = m / g.k;
    return b * g.R + g.nr + (m - b * g.k);
  }
  __device__ inline void store8(int m, int n, float (&v)[8]) const {
    const int b = m / g.k;
    const int p = g.ctx(st, b) + g.nr + (m - b * g.k);
    const size_t row = (size_t)srow(m);
    float pe[8];
    get8(pos + (size_t)p * d + n, pe);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += pe[i];
    if (temb) {
      get8(temb + (size_t)g.slot(b) * d + n, pe);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] += pe[i];
    }
    put8(X + row * d + n, v);
    if constexpr (sizeof(T) == 2) put8(Xh + row * d + n, v);
  }
};

// Q, K, V of a whole-sequence forward (the K-Forcing teacher rollout): GEMM
// row m = (b, i), i < n, in the layouts of the training-mask attention: Q
// [B][H][n][dh]; K and V [B][H][ldk][dh], row i at key koff + i.
template <typename T>
struct EpQKVSeq {
  T* Q;
  T* K;
  T* V;
  const float* bias;
  int n, ldk, koff, H, dh;
  int N, k, round;     // the round's row layout (positions of its rows)
  const float2* rope;  // rotary table, or null
  static constexpr bool kStats = false;
  __device__ inline int position(int i) const {
    const int nk = N * k;
    int q, base;
    if (round == 1) {
      if (i < N) return i;
      q = i - N;
      base = 1;
    } else {
      q = i < nk ? i : i - nk;
      base = i < nk ? 1 : 1 + k;
    }
    const int t = q / k;
    return t + base + (q - t * k);
  }
  __device__ inline void store8(int m, int c, float (&v)[8]) const {
    const int d = H * dh, which = c / d, cc = c - which * d, h = cc / dh, e = cc - h * dh;
    const int b = m / n, i = m - b * n;
    const size_t bh = (size_t)b * H + h;
    if (rope && which < 2) rotate8(v, rope, dh < 64 ? dh : 64, position(i), e);
    if (which == 0) put8(Q + (bh * n + i) * dh + e, v);
    else put8((which == 1 ? K : V) + (bh * ldk + koff + i) * dh + e, v);
  }
};

// Second noise-MLP layer of a whole-sequence forward: noise row m = (b, t, j)
// (N groups of k per sequence) lands in residual row b*n + off + t*k + j with
// the learned position t + shift + j added (the position of the token the
// row stands for) and, for a temperature-conditioned model, sequence b's
// temperature embedding.
template <typename T>
struct EpSeqNoise {
  float* X;
  T* Xh;
  const float* bias;
  const T* pos;
  const T* temb;  // [B][d] or null
  int n, off, N, k, shift, d;
  float2* lnst;
  static constexpr bool kStats = true;
  __device__ inline int cols() const { return d; }
  __device__ inline int srow(int m) const {
    const int nk = N * k, b = m / nk;
    return b * n + off + (m - b * nk);
  }
  __device__ inline void store8(int m, int c, float (&v)[8]) const {
    const int nk = N * k, b = m / nk, q = m - b * nk, t = q / k, j = q - t * k;
    const size_t row = (size_t)srow(m);
    float pe[8];
    get8(pos + (size_t)(t + shift + j) * d + c, pe);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += pe[i];
    if (temb) {
      get8(temb + (size_t)b * d + c, pe);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] += pe[i];
    }
    put8(X + row * d + c, v);
    if constexpr (sizeof(T) == 2) put8(Xh + row * d + c, v);
  }
};

// One K split of a split-K GEMM: fp32 C rows to part [M][ldp] (the kernel
// moves part to its split's slice); the bias and the GEMM's real epilogue run
// in splitk_reduce_kernel.
struct EpPartial {
  float* part;
  int ldp;
  const float* bias;  // always null: added by the reduction
  static constexpr bool kStats = false;
  __device__ inline void store8(int m, int n, float (&v)[8]) const {
    put8(part + (size_t)m * ldp + n, v);
  }
};

// Head: no store; per-tile argmax partials (and optional fp32 logits).
struct EpHead {
  static constexpr bool kStats = false;
  const float* bias;  // always null: the tied head has no bias
  float* pval;
  int* pidx;
  float* logits;
  int V;
  int n_tiles;
  // With st: the step's commit (C += nr, or per slot with a slot map) is done
  // by the first workgroup at its end.  No kernel of the step reads C after
  // the layers but the selection, which then takes C - nr; the commit saves
  // a launch per step.
  KfDevState* st = nullptr;
  KfStepGeom cg{};
  int cnr = 0;
};

// Head of a temperature-scaled sampling pass over every row (teacher
// targets): per (row, 128-column tile) the maximum M_t of the scaled logits
// x = l / tau_b and, per 16-column group q of the tile, sum exp(x - M_t) over
// the group's columns (< V).  Row m of this launch is row row0 + m of the step,
// sequence (row0 + m) / rows_per_seq.  logits (optional, fp32 [M][V]) keeps
// the unscaled logits.
struct EpHeadSample {
  static constexpr bool kStats = false;
  const float* bias;  // always null: the tied head has no bias
  float* pmax;        // [M][n_tiles]
  float* psub;        // [M][n_tiles][8]
  float* logits;
  const float* tau;   // [sequences]
  int row0, rows_per_seq, V, n_tiles;
  __device__ float inv_tau(int m) const {
    const float t = tau[(row0 + m) / rows_per_seq];
    return (t > 0.f && t < INFINITY) ? 1.0f / t : 1.0f;  // invalid tau: the select flags it
  }
};

template <typename Ep>
struct IsHead {
  static constexpr bool value = false;
};
template <>
struct IsHead<EpHead> {
  static constexpr bool value = true;
};
template <>
struct IsHead<EpHeadSample> {
  static constexpr bool value = true;
};

// ---------------------------------------------------------------- layout
// LDS tiles hold 8 16-byte chunks per row (one 128-byte K slab).  Chunk c of
// row r is stored at position c ^ ((r >> 1) & 7): sixteen lanes reading the
// same chunk of sixteen consecutive rows (one MFMA operand fetch) touch
// distinct 16-byte bank groups, and so do the 16-byte stores of a row.
constexpr int KCH = 8;
__device__ inline int swz(int r, int c) { return r * KCH + (c ^ ((r >> 1) & 7)); }

// Workgroups are dealt to the eight XCDs round-robin by linear id.  Each XCD
// gets a contiguous run of the tile order, and the order walks the grid in
// column groups of kGroupN weight tiles, row by row inside a group (the
// group's columns fastest): the workgroups an XCD runs together then cover a
// compact block of rows and columns, so both operand strips stay in that
// XCD's L2 instead of every XCD streaming all of A once per weight strip.
// Groups of 8 measured best (against 2, 4, 12, 16 and 32: LM1B-shaped batch
// 64 +1.7 % over 4, OWT-shaped batch 512 +0.9 %, the 24-layer backbone
// +0.3 %).
constexpr int kGroupN = 8;
__device__ inline void tile_coords(int lin, int gm, int gn, int& tm, int& tn) {
  const int total = gm * gn;
  const int q = total >> 3, r = total & 7;
  const int x = lin & 7, j = lin >> 3;
  const int t = x * q + (x < r ? x : r) + j;  // this XCD's run of the order
  const int grp = t / (gm * kGroupN), first = grp * kGroupN;
  const int width = gn - first < kGroupN ? gn - first : kGroupN;
  const int u = t - grp * gm * kGroupN;
  tm = u / width;
  tn = first + u % width;
}

// Which A row feeds GEMM row m (MODE 0: row m; 1: noise row m of the step;
// 2: last real row of sequence m).
template <int MODE>
__device__ inline int map_row(int m, const KfStepGeom& g) {
  if constexpr (MODE == 1) return (m / g.k) * g.R + g.nr + (m % g.k);
  else if constexpr (MODE == 2) return m * g.R + g.nr - 1;
  else return m;
}

// A operand: a compute-dtype matrix [arows][lda], rows picked by map_row.
// With NORM, the GEMM applies the LayerNorm of each A row through the folded
// weights: W' = W diag(g) (scaled at weight load), c1 = W' 1, c2 = W beta, so
//   LN(x) W^T = rstd * (x W'^T - mu * c1) + c2,
// where mu and rstd = 1 / sqrt(var + 1e-5) come from the row's partial sums
// lnst [arows][K / 16] (sum x, sum x^2 per 16 columns of the fp32 residual
// row), written by the kernel that produced the row.
struct GemmA {
  const void* A;
  int lda;
  int arows;
  const float* c1;
  const float* c2;
  const float2* lnst;
  KfStepGeom g;
  int rms;  // RMSNorm statistics (mu = 0)
};

// ---------------------------------------------------------------- kernel
// S-stage LDS ring fed by direct-to-LDS loads, with a register double buffer
// of MFMA operands (pipeline described at the K loop).  Each wavefront loads
// 8 rows (one 128-byte slab each) per instruction: BM / (8 NWV) A instructions
// and BN / (8 NWV) W instructions per stage for NWV wavefronts.  The 128 x 128
// and 64 x 128 body tiles run eight wavefronts (64 x 32 and 32 x 32 per
// wavefront), held to four wavefronts per SIMD (at most 128 registers) so that
// two workgroups share a CU: that hides the ring's barrier and LDS latencies
// better than four wavefronts with twice the per-wavefront tile (measured
// 3-12 % faster per GEMM at M = 512 to 4096, the results bit for bit the same;
// with 146 registers the folded-norm 128 x 128 tile fitted one workgroup per
// CU and was 23 % slower than with four wavefronts).  With KG = 2 the
// workgroup holds two such groups of WM x WN wavefronts, each with a ring of
// its own over half of the K steps; the second group's sums are added to the
// first's through LDS before the epilogue (grids of at most one workgroup per
// CU, where the two rings double the operand loads in flight).
template <typename T, int BM, int BN, int WM, int WN, int S, int MODE, bool NORM, class Ep,
          int KG = 1>
__global__ void __launch_bounds__(64 * WM * WN * KG)
    __attribute__((amdgpu_waves_per_eu(WM * WN * KG == 8 ? 4 : 1)))
    gemm_kernel(GemmA ga, const T* __restrict__ W, int ldw, int M, int N, int K, Ep ep,
                int ksplit) {
  constexpr int CH = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  constexpr int BK = KCH * CH;             // K per slab
  constexpr int MW = BM / WM, NW = BN / WN;
  constexpr int TM = MW / 16, TN = NW / 16;
  constexpr int NWV = WM * WN;                // wavefronts of one K group
  constexpr int NT = 64 * NWV * KG;           // threads
  constexpr int RPI = 8 * NWV;                // rows one DMA instruction round covers
  constexpr int PA = BM / RPI, PW = BN / RPI, PER = PA + PW;
  constexpr int ROWB = KCH * 16;                 // bytes per staged row
  static_assert(NWV == 4 || NWV == 8, "four or eight wavefronts");
  static_assert(MW % 16 == 0 && NW % 16 == 0, "16x16 MFMA tiles");
  static_assert(BM % RPI == 0 && BN % RPI == 0, "whole DMA instructions per wavefront");
  static_assert(S >= 2 && S <= 8, "ring depth");
  static_assert((S - 1) * PER < 64, "vmcnt range");
  static_assert(KG == 1 || KG == 2, "one or two K groups");
  static_assert(KG == 1 || !IsHead<Ep>::value, "K groups: not with the head epilogues");

  __shared__ u32x4 sbuf[KG][S][(BM + BN) * KCH];
  __shared__ float2 sStat[NORM ? BM : 1];

  const int tid = threadIdx.x, lane = tid & 63;
  // K group kg (of KG) runs its own ring over its share of the K steps;
  // wave is the wavefront's index inside its group.
  const int kg = KG == 1 ? 0 : (tid >> 6) / NWV;
  const int wave = KG == 1 ? tid >> 6 : (tid >> 6) % NWV;
  const int wm = wave / WN, wn = wave % WN;
  const int gm = (M + BM - 1) / BM, gn = (N + BN - 1) / BN;
  // ksplit > 1 only with EpPartial: workgroup (tile, split) takes K steps
  // [split * nk, (split + 1) * nk) and writes its own slice of the parts.
  const int split = (int)blockIdx.x % ksplit;
  int tmi, tni;
  tile_coords((int)blockIdx.x / ksplit, gm, gn, tmi, tni);
  const int m0 = tmi * BM, n0 = tni * BN;
  const int nk = K / BK / ksplit / KG;  // K steps of this wavefront's group
  const int kbeg = (split * KG + kg) * nk;
  if constexpr (std::is_same<Ep, EpPartial>::value) ep.part += (size_t)split * M * ep.ldp;

  const T* A = static_cast<const T*>(ga.A);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, (uint32_t)((size_t)ga.arows * ga.lda * sizeof(T)));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(W, (uint32_t)((size_t)N * ldw * sizeof(T)));

  // DMA sources at k = 0.  Lane l of a load covers row r0 + l / 8 and LDS
  // slot l % 8, which holds chunk (l % 8) ^ ((r >> 1) & 7) of the row: the
  // swizzled layout of swz().  Rows past the end re-read the last row: such a
  // row only feeds its own output row, which is never stored.
  uint32_t aoff[PA], woff[PW];
#pragma unroll
  for (int j = 0; j < PA; ++j) {
    const int r = wave * 8 + RPI * j + lane / 8, c = (lane & 7) ^ ((r >> 1) & 7);
    const int gr = m0 + r < M ? m0 + r : M - 1;
    aoff[j] = (uint32_t)(((size_t)map_row<MODE>(gr, ga.g) * ga.lda + c * CH) * sizeof(T));
  }
#pragma unroll
  for (int j = 0; j < PW; ++j) {
    const int r = wave * 8 + RPI * j + lane / 8, c = (lane & 7) ^ ((r >> 1) & 7);
    const int gr = n0 + r < N ? n0 + r : N - 1;
    woff[j] = (uint32_t)(((size_t)gr * ldw + c * CH) * sizeof(T));
  }
  auto issue = [&](int stage, int kt) {
    const uint32_t so = (uint32_t)((kbeg + kt) * BK * (int)sizeof(T));
#pragma unroll
    for (int j = 0; j < PA; ++j) dma16(ra, aoff[j], so, &sbuf[kg][stage][(wave * 8 + RPI * j) * KCH]);
#pragma unroll
    for (int j = 0; j < PW; ++j)
      dma16(rw, woff[j], so, &sbuf[kg][stage][(BM + wave * 8 + RPI * j) * KCH]);
  };

  // LDS read offsets within a stage.  Every row a lane reads is congruent to
  // lane % 16 modulo 16, so one swizzle key serves all of them.
  const int key = (lane & 15) >> 1;
  uint32_t rdA[2], rdW[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int ch = (s * 4 + (lane >> 4)) ^ key;
    rdA[s] = (uint32_t)(((wm * MW + (lane & 15)) * KCH + ch) * 16);
    rdW[s] = (uint32_t)(((BM + wn * NW + (lane & 15)) * KCH + ch) * 16);
  }
  f32x4 acc[TN][TM];
#pragma unroll
  for (int x = 0; x < TN; ++x)
#pragma unroll
    for (int y = 0; y < TM; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Column constants of this lane's output columns (bias; folded-LayerNorm
  // sums), loaded now so that the epilogue does not wait on memory.
  f32x4 pb[TN], p1[TN], p2[TN];
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) {
    const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
    const int nc = n < N ? n : 0;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    pb[tn] = ep.bias ? *reinterpret_cast<const f32x4*>(ep.bias + nc) : z;
    p1[tn] = NORM ? *reinterpret_cast<const f32x4*>(ga.c1 + nc) : z;
    p2[tn] = NORM ? *reinterpret_cast<const f32x4*>(ga.c2 + nc) : z;
  }

  // One 32-wide K slice (half a slab) of this wavefront's operands.
  struct Slice {
    u32x4 a[TN];  // weight rows (MFMA "A")
    u32x4 b[TM];  // activation rows (MFMA "B")
  };
  auto read_slice = [&](int stage, int s, Slice& f) {
    const uint32_t sb = lds_addr(&sbuf[kg][stage][0]);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) f.a[tn] = ds_read16(sb + rdW[s] + tn * 16 * ROWB);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) f.b[tm] = ds_read16(sb + rdA[s] + tm * 16 * ROWB);
  };
  auto pin_slice = [&](Slice& f) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) pin(f.a[tn]);
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) pin(f.b[tm]);
  };
  auto mma_slice = [&](const Slice& f) {
#pragma unroll
    for (int tn = 0; tn < TN; ++tn)
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) Mfma<T>::mma(f.a[tn], f.b[tm], acc[tn][tm]);
  };
  // Software pipeline over K steps (one 64-wide slab per step, two slices):
  //   [slice 0 of step kt is in registers]
  //   read slice 1 of step kt; MFMAs of slice 0
  //   wait for the reads; wait for this wavefront's loads of stage kt + 1
  //   barrier: stage kt + 1 has landed, every read of stage kt is done
  //   load step kt + S into stage kt's buffer; read slice 0 of step kt + 1
  //   MFMAs of slice 1 of step kt; wait for the reads
  // so LDS reads always run under MFMAs, and S stages are loading at a time.
  // Folded LayerNorm: each row's mean and rstd from its partial sums.  The
  // partials are loaded before the operand loads are issued (so waiting for
  // them does not wait for the operands) and reduced by the TPR consecutive
  // lanes that share a row.
  static_assert(!NORM || NT % BM == 0, "whole threads per row for the statistics");
  constexpr int TPR = NORM ? NT / BM : 1;
  // float4 loads (two partials each) per lane, unrolled: whole rows up to
  // K = 1024; wider rows finish in a loop.
  constexpr int PMAX = NORM ? (32 / TPR > 0 ? 32 / TPR : 1) : 1;
  float4 part[PMAX];
  const int parts4 = K / 32;  // float4 words per row
  const float4* prow = nullptr;
  // The prologue is straight-line code: the partial loads (indices clamped to
  // the row, extra words masked below) and the first S stages are issued
  // unconditionally, so the compiler's wait before the statistics covers the
  // partials only.  Behind a branch it waits for every load in flight, the
  // whole ring included.  A stage past this split's K range reads bytes that
  // are never consumed (the buffer range returns zeros past its end), and it
  // has landed before the first barrier.
  if constexpr (NORM) {
    const int r = tid / TPR, gr = m0 + r < M ? m0 + r : M - 1;
    prow = reinterpret_cast<const float4*>(ga.lnst + (size_t)map_row<MODE>(gr, ga.g) * (K / 16));
#pragma unroll
    for (int j = 0; j < PMAX; ++j) {
      const int w = (tid % TPR) + j * TPR;
      part[j] = prow[w < parts4 ? w : parts4 - 1];
    }
  }
  // A residual epilogue's old values for the chunks this thread will store
  // (one per epilogue band when a band takes one chunk pass), loaded before the
  // operand stages so that the epilogue does not wait a memory round trip per
  // band.  Loads complete in issue order, so the stage waits below still hold.
  // Four-wavefront tiles only (steps of up to 512 rows: LM1B batch 64 +0.7 %,
  // OWT-shaped batch 16 +1.2 %); the eight-wavefront 64 x 128 tile of the
  // large batches measured 0.3 % slower with it.
  constexpr int ECPR = BN / 8, ENCH = (MW * ECPR + NT - 1) / NT;
  constexpr bool kPre = HasPre<Ep>::value && !IsHead<Ep>::value && NWV == 4 && WM * ENCH <= 2;
  float xpre[kPre ? WM * ENCH : 1][8];
  if constexpr (kPre) {
#pragma unroll
    for (int p = 0; p < WM; ++p)
#pragma unroll
      for (int it = 0; it < ENCH; ++it) {
        const int c0 = it * NT + tid, c = c0 < MW * ECPR ? c0 : MW * ECPR - 1;
        const int m = m0 + p * MW + c / ECPR, n = n0 + (c % ECPR) * 8;
        ep.pre8(m < M ? m : M - 1, n < N ? n : 0, xpre[p * ENCH + it]);
      }
  }
  Slice f0, f1;
#pragma unroll
  for (int i = 0; i < S; ++i) issue(i, i);
  if constexpr (NORM) {
    // the row's mean from the group sums, then the merged squared deviations
    float a = 0.f;
#pragma unroll
    for (int j = 0; j < PMAX; ++j)
      a += (tid % TPR) + j * TPR < parts4 ? part[j].x + part[j].z : 0.f;
    for (int w = (tid % TPR) + PMAX * TPR; w < parts4; w += TPR) {  // K > 1024 only
      const float4 v = prow[w];
      a += v.x + v.z;
    }
#pragma unroll
    for (int off = 1; off < TPR; off <<= 1) a += __shfl_xor(a, off, 64);
    const float mu = ga.rms ? 0.f : a / (float)K;
    float b = 0.f;
#pragma unroll
    for (int j = 0; j < PMAX; ++j) {
      const float q = ln_group_sq(make_float2(part[j].x, part[j].y), mu) +
                      ln_group_sq(make_float2(part[j].z, part[j].w), mu);
      b += (tid % TPR) + j * TPR < parts4 ? q : 0.f;
    }
    for (int w = (tid % TPR) + PMAX * TPR; w < parts4; w += TPR) {
      const float4 v = prow[w];
      b += ln_group_sq(make_float2(v.x, v.y), mu) + ln_group_sq(make_float2(v.z, v.w), mu);
    }
#pragma unroll
    for (int off = 1; off < TPR; off <<= 1) b += __shfl_xor(b, off, 64);
    if (tid % TPR == 0) sStat[tid / TPR] = make_float2(mu, 1.0f / sqrtf(b / (float)K + 1e-5f));
  }
  if (nk > S - 1) vm_wait<(S - 1) * PER>();
  else vm_wait<0>();
  lgkm_wait0();  // sStat written before the barrier publishes it
  __builtin_amdgcn_s_barrier();
  read_slice(0, 0, f0);
  lgkm_wait0();
  pin_slice(f0);
  for (int kt0 = 0; kt0 < nk; kt0 += S) {
#pragma unroll
    for (int i = 0; i < S; ++i) {
      const int kt = kt0 + i;
      if (kt < nk) {
        read_slice(i, 1, f1);
        __builtin_amdgcn_sched_barrier(0);  // the reads issue first,
        mma_slice(f0);                       // the MFMAs run under them,
        __builtin_amdgcn_sched_barrier(0);  // and only then the wait
        lgkm_wait0();
        pin_slice(f1);
        if (kt + 1 < nk) {
          if (kt + S - 1 < nk) vm_wait<(S - 2) * PER>();
          else vm_wait<0>();
          __builtin_amdgcn_s_barrier();
          if (kt + S < nk) issue(i, kt + S);
          read_slice((i + 1) % S, 0, f0);
        }
        __builtin_amdgcn_sched_barrier(0);
        mma_slice(f1);
        __builtin_amdgcn_sched_barrier(0);
        lgkm_wait0();
        pin_slice(f0);
      }
    }
  }
  if constexpr (KG == 2) {
    // Group 1's sums (the second half of K) are added to group 0's through
    // LDS: the same order as a two-way split summed by the reduction kernel.
    float4* xch = reinterpret_cast<float4*>(&sbuf[1][0][0]);
    static_assert(NWV * TN * TM * 64 * 16 <= S * (BM + BN) * KCH * 16, "exchange fits the ring");
    __syncthreads();  // both rings are read out
    if (kg == 1) {
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const f32x4 v = acc[tn][tm];
          xch[((wave * TN + tn) * TM + tm) * 64 + lane] = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
    __syncthreads();
    if (kg == 0) {
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm) {
          const float4 v = xch[((wave * TN + tn) * TM + tm) * 64 + lane];
          acc[tn][tm][0] += v.x;
          acc[tn][tm][1] += v.y;
          acc[tn][tm][2] += v.z;
          acc[tn][tm][3] += v.w;
        }
    }
  }

  // Folded LayerNorm (if any) and bias for 16x16 tile (tn, tm).  The row
  // statistics of this lane's TM rows are read from LDS once, here.
  float2 rst[NORM ? TM : 1];
  if constexpr (NORM) {
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) rst[tm] = sStat[wm * MW + tm * 16 + (lane & 15)];
  }
  auto apply = [&](f32x4 v, int tm, int tn) -> f32x4 {
    f32x4 r;
    if constexpr (NORM) {
      const float2 st = rst[tm];
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = st.y * (v[i] - st.x * p1[tn][i]) + p2[tn][i] + pb[tn][i];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = v[i] + pb[tn][i];
    }
    return r;
  };

  if constexpr (!IsHead<Ep>::value) {
    // Stores through LDS: one wavefront row band (MW rows) at a time is
    // written to the free ring as fp32 rows padded by 16 bytes (the 16 lanes
    // of a column write then hit distinct banks) and read back as 8-column
    // row chunks, consecutive lanes taking consecutive chunks.
    constexpr int SROW = BN + 4;  // fp32 words per staged row
    constexpr int CPR = BN / 8;   // chunks per row
    static_assert(MW * SROW * 4 <= S * (BM + BN) * KCH * 16, "staging fits the ring");
    static_assert((MW * CPR) % 64 == 0, "whole wavefronts per chunk pass");
    float* stage = reinterpret_cast<float*>(&sbuf[0][0][0]);
    __syncthreads();  // every wavefront is done reading the ring
#pragma unroll
    for (int pass = 0; pass < WM; ++pass) {
      if (kg == 0 && wm == pass) {
#pragma unroll
        for (int tn = 0; tn < TN; ++tn)
#pragma unroll
          for (int tm = 0; tm < TM; ++tm) {
            const f32x4 r = apply(acc[tn][tm], tm, tn);
            float* q = stage + (tm * 16 + (lane & 15)) * SROW + wn * NW + tn * 16 + 4 * (lane >> 4);
            *reinterpret_cast<float4*>(q) = make_float4(r[0], r[1], r[2], r[3]);
          }
      }
      __syncthreads();
      bool by_column = false;
      if constexpr (HasColumns<Ep>::value) by_column = ep.column_tile(n0);
#pragma unroll
      for (int c0 = 0; c0 < MW * CPR; c0 += NT) {
        const int c = c0 + tid;
        if constexpr (HasColumns<Ep>::value) {
          if (by_column) {  // 8 consecutive rows of one column per lane
            static_assert(MW % 8 == 0, "whole 8-row groups per band");
            if (c0 + NT <= MW * CPR || c < MW * CPR) {
              const int cg = c / BN, cl = c % BN;
              const int m = m0 + pass * MW + cg * 8, n = n0 + cl;
              float v[8];
#pragma unroll
              for (int r = 0; r < 8; ++r) v[r] = stage[(cg * 8 + r) * SROW + cl];
              if (m < M && n < N) ep.store_col8(m, n, v, M);
            }
            continue;
          }
        }
        if (c0 + NT <= MW * CPR || c < MW * CPR) {
          const int rr = c / CPR, cc = c % CPR;
          const int m = m0 + pass * MW + rr, n = n0 + cc * 8;
          const bool live = m < M && n < N;
          float v[8];
          const float4 lo = *reinterpret_cast<const float4*>(stage + rr * SROW + cc * 8);
          const float4 hi = *reinterpret_cast<const float4*>(stage + rr * SROW + cc * 8 + 4);
          v[0] = lo.x; v[1] = lo.y; v[2] = lo.z; v[3] = lo.w;
          v[4] = hi.x; v[5] = hi.y; v[6] = hi.z; v[7] = hi.w;
          if constexpr (kPre) {
            if (live) ep.store8_pre(m, n, v, xpre[pass * ENCH + c0 / NT]);
          } else {
            if (live) ep.store8(m, n, v);
          }
          if constexpr (Ep::kStats) {
            // chunks 2j and 2j + 1 of a row (lanes c, c ^ 1) form 16-column group j
            const float2 gs = ln_group16(v);
            if (live && (cc & 1) == 0) ep.lnst[(size_t)ep.srow(m) * (ep.cols() / 16) + n / 16] = gs;
          }
        }
      }
      __syncthreads();  // the next band reuses the staging rows
    }
  } else if constexpr (std::is_same<Ep, EpHeadSample>::value) {
    // Tile maximum of the scaled logits per row (lane-local, across the four
    // lane groups holding the row, then across the WN wavefronts), then the
    // 16-column group sums of exp(x - M_t): group (wn, tn) is exactly the
    // 16 columns that the four lane groups of wavefront wn hold for tn.
    static_assert(BN == 128 && WN * TN == 8, "eight 16-column groups per head tile");
    __shared__ float redm[WN][BM];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int mloc = wm * MW + tm * 16 + (lane & 15);
      const int m = m0 + mloc;
      const float it = ep.inv_tau(m < M ? m : 0);
      float bv = -INFINITY;
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
        const f32x4 v = apply(acc[tn][tm], tm, tn);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (n + i < ep.V) bv = fmaxf(bv, v[i] * it);
      }
      bv = fmaxf(bv, __shfl_xor(bv, 16, 64));
      bv = fmaxf(bv, __shfl_xor(bv, 32, 64));
      if ((lane >> 4) == 0) redm[wn][mloc] = bv;
    }
    __syncthreads();
    const int nt = n0 / BN;
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) {
      const int mloc = wm * MW + tm * 16 + (lane & 15);
      const int m = m0 + mloc;
      const float it = ep.inv_tau(m < M ? m : 0);
      float mt = redm[0][mloc];
#pragma unroll
      for (int w = 1; w < WN; ++w) mt = fmaxf(mt, redm[w][mloc]);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) {
        const int n = n0 + wn * NW + tn * 16 + 4 * (lane >> 4);
        const f32x4 v = apply(acc[tn][tm], tm, tn);
        float sg = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (n + i < ep.V) sg += __expf(v[i] * it - mt);
        sg += __shfl_xor(sg, 16, 64);
        sg += __shfl_xor(sg, 32, 64);
        if (m < M) {
          if ((lane >> 4) == 0) ep.psub[((size_t)m * ep.n_tiles + nt) * 8 + wn * TN + tn] = sg;
          if (ep.logits) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (n + i < ep.V) ep.logits[(size_t)m * ep.V + n + i] = v[i];
          }
        }
      }
      if (m < M && wn == 0 && (lane >> 4) == 0) ep.pmax[(size_t)m * ep.n_tiles + nt] = mt;
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
        const f32x4 v = apply(acc[tn][tm], tm, tn);
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
    if (ep.st && blockIdx.x == 0) {
      if (ep.cg.map) {
        for (int b = tid; b < ep.cg.B; b += NT) ep.cg.cs[ep.cg.map[b]] += ep.cnr;
      } else if (tid == 0) {
        ep.st->C += ep.cnr;
      }
    }
  }
}

// ------------------------------------------------------- skinny GEMM
// Steps of at most 16 rows (decode blocks of one to four sequences, the AR
// baseline at small batch) do little arithmetic per weight byte, and the tiled
// kernel's K loop then runs at the latency of its LDS ring and barriers.  Here
// one workgroup takes 16 output columns and its KW wavefronts split K: each
// wavefront streams its K range of the 16 weight rows and of the (at most 16)
// activation rows from memory straight into MFMA operands (16-byte chunks, the
// same chunk-to-k assignment on both sides, up to 2U K steps of loads in
// flight, no LDS and no barrier in the loop).  The wavefronts' partial sums meet in LDS
// in wavefront order, and the 16 x 16 tile goes through the folded LayerNorm,
// the bias and the same epilogues as the tiled kernel.
template <typename T, int KW, int MODE, bool NORM, class Ep>
__global__ void __launch_bounds__(64 * KW)
    gemm_skinny_kernel(GemmA ga, const T* __restrict__ W, int ldw, int M, int N, int K, Ep ep) {
  static_assert(sizeof(T) == 2, "16-bit operands (one 16x16x32 MFMA per K step)");
  static_assert(KW >= 4, "at least one thread per tile element");
  constexpr int U = KW >= 16 ? 4 : 8;  // 32-wide K steps per batch of loads
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int kw = K / KW, steps = kw / 32;
  const T* A = static_cast<const T*>(ga.A);

  // Folded LayerNorm: the row partial sums of the 16 rows (16 threads per
  // row) are loaded first and reduced once the operand loads are in flight,
  // so both wait on one memory round trip.
  // Every prologue load is unconditional, its index clamped into range (the
  // extra values are masked where they are used): a load behind a branch makes
  // the compiler wait for all loads in flight at the join.
  constexpr int PS = 4;  // partial sums per thread held in registers (K <= 1024)
  __shared__ float2 sStat[16];
  float2 ps[PS];
  const float2* pr = nullptr;
  if constexpr (NORM) {
    const int pm = (tid >> 4) & 15;  // threads past 256 repeat rows 0..15; only the first 256 use them
    pr = ga.lnst + (size_t)map_row<MODE>(pm < M ? pm : M - 1, ga.g) * (K / 16);
#pragma unroll
    for (int i = 0; i < PS; ++i) {
      const int w = (tid & 15) + 16 * i;
      ps[i] = pr[w < K / 16 ? w : K / 16 - 1];
    }
  }
  // The column constants of this thread's tile element (bias, folded-norm
  // sums) and a residual-stream epilogue's old values are loaded now as well.
  const int ec = tid & 15, en = n0 + ec < N ? n0 + ec : N - 1;
  float e_pb = 0.f, e_c1 = 0.f, e_c2 = 0.f;
  if (tid < 256) {
    if (ep.bias) e_pb = ep.bias[en];
    if constexpr (NORM) {
      e_c1 = ga.c1[en];
      e_c2 = ga.c2[en];
    }
  }
  const int sm = (lane >> 1) & 15, scc = lane & 1, sn = n0 + 8 * scc;
  const bool slive = wave == 0 && lane < 32 && sm < M && sn < N;
  float pre[8];
  if constexpr (HasPre<Ep>::value) {
    if (slive) ep.pre8(sm, sn, pre);
  }

  // Lane (r, q) feeds weight row n0 + r and activation row r, elements
  // 8q .. 8q + 7 of each 32-wide K step.  Rows past the end re-read the last
  // row: their outputs are never stored.
  const int wrow = n0 + r < N ? n0 + r : N - 1;
  const int arow = map_row<MODE>(r < M ? r : M - 1, ga.g);
  const u32x4* pw = reinterpret_cast<const u32x4*>(W + (size_t)wrow * ldw + wave * kw + 8 * q);
  const u32x4* pa = reinterpret_cast<const u32x4*>(A + (size_t)arow * ga.lda + wave * kw + 8 * q);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  // Two named load batches alternate (no register copies between them, which
  // would wait for loads still in flight): batch B loads while batch A feeds
  // the MFMAs, and the other way round.
  u32x4 wa[U], xa[U], wb[U], xb[U];
  // Four wavefronts (one batch covers a K range of up to 8 steps): steps past
  // the end load an earlier step instead (valid memory, and a different
  // address from every other load of the batch: loads of one address would be
  // merged into one and copied, and a copy waits for its load), so the batch
  // is straight-line code.  Sixteen wavefronts (two batches of 4, six steps)
  // keep zero-filled loads behind the step bound: with the straight-line form
  // the compiler made each load of the second batch wait for the first batch
  // (MLP-down at batch 1: 7.6 -> 9.0 us).  mma() skips the steps past the end.
  auto load = [&](u32x4 (&w)[U], u32x4 (&x)[U], int s0) {
#pragma unroll
    for (int i = 0; i < U; ++i) {
      if constexpr (KW >= 16) {
        const int t = s0 + i;
        const u32x4 z = {0u, 0u, 0u, 0u};
        w[i] = t < steps ? pw[4 * t] : z;
        x[i] = t < steps ? pa[4 * t] : z;
      } else {
        const int t = s0 + i < steps ? s0 + i : (s0 + i) % steps;
        w[i] = pw[4 * t];
        x[i] = pa[4 * t];
      }
    }
  };
  auto mma = [&](const u32x4 (&w)[U], const u32x4 (&x)[U], int s0) {
#pragma unroll
    for (int i = 0; i < U; ++i)
      if (s0 + i < steps) Mfma<T>::mma(w[i], x[i], acc);
  };
  load(wa, xa, 0);
  if constexpr (NORM) {
    if (tid < 256) {
      // the row's mean from the group sums, then the merged squared deviations
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < PS; ++i) a += (tid & 15) + 16 * i < K / 16 ? ps[i].x : 0.f;
      for (int w = (tid & 15) + 16 * PS; w < K / 16; w += 16) a += pr[w].x;  // K > 1024 only
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) a += __shfl_xor(a, off, 64);
      const float mu = ga.rms ? 0.f : a / (float)K;
      float b = 0.f;
#pragma unroll
      for (int i = 0; i < PS; ++i) b += (tid & 15) + 16 * i < K / 16 ? ln_group_sq(ps[i], mu) : 0.f;
      for (int w = (tid & 15) + 16 * PS; w < K / 16; w += 16) b += ln_group_sq(pr[w], mu);
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) b += __shfl_xor(b, off, 64);
      if ((tid & 15) == 0) sStat[tid >> 4] = make_float2(mu, 1.0f / sqrtf(b / (float)K + 1e-5f));
    }
  }
  for (int s = 0; s < steps; s += 2 * U) {
    if (s + U < steps) load(wb, xb, s + U);
    mma(wa, xa, s);
    if (s + U >= steps) break;
    if (s + 2 * U < steps) load(wa, xa, s + 2 * U);
    mma(wb, xb, s + U);
  }

  // This lane holds row r, columns 4q .. 4q + 3 of its wavefront's K range.
  constexpr int SR = 20;  // padded row of the 16 x 16 tile, in floats
  __shared__ __align__(16) float sred[KW][16 * SR];
  __shared__ float sout[16 * SR];
  *reinterpret_cast<float4*>(&sred[wave][r * SR + 4 * q]) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  __syncthreads();
  if (tid < 256) {  // one tile element per thread: sum over K ranges, norm, bias
    const int m = tid >> 4, c = ec;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < KW; ++w) v += sred[w][m * SR + c];
    if constexpr (NORM) {
      const float2 st = sStat[m];
      v = st.y * (v - st.x * e_c1) + e_c2 + e_pb;
    } else {
      v = v + e_pb;
    }
    sout[m * SR + c] = v;
  }
  __syncthreads();
  if (wave != 0) return;
  if constexpr (HasColumns<Ep>::value) {
    if (ep.column_tile(n0)) {  // 8 consecutive rows of one column per lane
      const int cg = lane >> 4, cl = lane & 15;
      const int m = 8 * cg, n = n0 + cl;
      if (lane < 32 && m < M && n < N) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = sout[(m + i) * SR + cl];
        ep.store_col8(m, n, v, M);
      }
      return;
    }
  }
  const int m = sm, cc = scc, n = sn;
  const bool live = slive;
  float v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = sout[m * SR + 8 * cc + i];
  if constexpr (HasPre<Ep>::value) {
    if (live) ep.store8_pre(m, n, v, pre);
  } else {
    if (live) ep.store8(m, n, v);
  }
  if constexpr (Ep::kStats) {
    // chunks 0 and 1 of a row (lanes 2j, 2j + 1) form its 16-column group
    const float2 gs = ln_group16(v);
    if (live && cc == 0) ep.lnst[(size_t)ep.srow(m) * (ep.cols() / 16) + n / 16] = gs;
  }
}

template <typename T, int MODE, bool NORM, class Ep>
hipError_t launch_skinny(const GemmA& ga, const T* W, int M, int N, int K, const Ep& ep,
                         hipStream_t s) {
  if (K % 512 == 0 && K >= 2048)  // long K (MLP-down): sixteen wavefronts of 6+ K steps
    launch((gemm_skinny_kernel<T, 16, MODE, NORM, Ep>), dim3(N / 16), dim3(1024), 0, s, ga, W, K,
           M, N, K, ep);
  else
    launch((gemm_skinny_kernel<T, 4, MODE, NORM, Ep>), dim3(N / 16), dim3(256), 0, s, ga, W, K, M,
           N, K, ep);
  return hipGetLastError();
}

template <typename T, int BM, int BN, int WM, int WN, int S, int MODE, bool NORM, int KG = 1,
          class Ep>
hipError_t launch_tile(const GemmA& ga, const T* W, int ldw, int M, int N, int K, const Ep& ep,
                       hipStream_t s, int ksplit = 1) {
  const int tiles = ((N + BN - 1) / BN) * ((M + BM - 1) / BM);
  launch((gemm_kernel<T, BM, BN, WM, WN, S, MODE, NORM, Ep, KG>), dim3(tiles * ksplit),
                     dim3(64 * WM * WN * KG), 0, s, ga, W, ldw, M, N, K, ep, ksplit);
  return hipGetLastError();
}

// Reduction of a split-K GEMM: C = sum of the parts in split order, plus the
// bias, through the GEMM's epilogue (and its LayerNorm partial sums).  One
// thread per 8-column chunk of a row.  The split count is a template
// parameter so that every load (the parts, a residual epilogue's old row, the
// bias) is issued before the first is waited for: one memory round trip.
template <int NS, class Ep>
__global__ void __launch_bounds__(128)
    splitk_reduce_kernel(const float* __restrict__ part, int M, int N, Ep ep) {
  const int m = blockIdx.x, c = blockIdx.y * 128 + threadIdx.x, n = c * 8;
  const bool live = n < N;
  const int nc = live ? n : 0;  // past-the-end threads load column 0 and store nothing
  float x[NS][8];
#pragma unroll
  for (int sp = 0; sp < NS; ++sp) get8(part + ((size_t)sp * M + m) * N + nc, x[sp]);
  float pre[8];
  if constexpr (HasPre<Ep>::value) ep.pre8(m, nc, pre);
  float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (ep.bias) {
#pragma unroll
    for (int i = 0; i < 8; ++i) bv[i] = ep.bias[nc + i];
  }
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sp = 0; sp < NS; ++sp)
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += x[sp][i];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] += bv[i];
  if (live) {
    if constexpr (HasPre<Ep>::value) ep.store8_pre(m, n, v, pre);
    else ep.store8(m, n, v);
  }
  if constexpr (Ep::kStats) {
    const float2 gs = ln_group16(v);
    if (live && (c & 1) == 0) ep.lnst[(size_t)ep.srow(m) * (ep.cols() / 16) + n / 16] = gs;
  }
}

template <class Ep>
hipError_t launch_splitk_reduce(const float* part, int splits, int M, int N, const Ep& ep,
                                hipStream_t s) {
  const dim3 grid(M, (N / 8 + 127) / 128), block(128);
  switch (splits) {
    case 2: launch(splitk_reduce_kernel<2, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 3: launch(splitk_reduce_kernel<3, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 4: launch(splitk_reduce_kernel<4, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 6: launch(splitk_reduce_kernel<6, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 8: launch(splitk_reduce_kernel<8, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 12: launch(splitk_reduce_kernel<12, Ep>, grid, block, 0, s, part, M, N, ep); break;
    case 16: launch(splitk_reduce_kernel<16, Ep>, grid, block, 0, s, part, M, N, ep); break;
    default: return hipErrorInvalidValue;  // launch_plain picks only the counts above
  }
  return hipGetLastError();
}

// A GEMM without a folded LayerNorm whose grid cannot fill the chip and whose
// K is long (24 K steps or more) is run as K splits (up to 16, at least two K
// steps each, about 320 workgroups in all) into the fp32 workspace, then
// reduced.  Short-K grids do not split: on the OWT-shaped model the
// out-projection (K = 768) at batch 8 and 16 took 15 instead of 22.5 ms per
// generate without its split and reduction kernel (whole generate +2.5 %).
// Plain GEMM grids of this many tiles take two K groups per workgroup: from
// half a workgroup per CU to one.  Smaller grids take them only when K is too
// short for a split across workgroups (the K = 768 out-projection at
// OWT-shaped batch 4 to 32: +1.0 %, +0.8 %, +0.3 %, 0 %); with the long-K
// MLP-down as well they measured mixed (batch 4 +2.6 %, batch 16 -1.2 %).
constexpr int kTwoGroupMin = 128, kTwoGroupMax = 256;

template <typename T, int BM, int BN, int WM, int WN, int S, int KG, class Ep>
hipError_t launch_tile_kg(int kg, const GemmA& ga, const T* W, int M, int N, int K, const Ep& ep,
                          hipStream_t s, int ksplit) {
  if constexpr (KG == 2) {
    if (kg == 2) return launch_tile<T, BM, BN, WM, WN, S, 0, false, 2>(ga, W, K, M, N, K, ep, s, ksplit);
  }
  return launch_tile<T, BM, BN, WM, WN, S, 0, false>(ga, W, K, M, N, K, ep, s, ksplit);
}

template <typename T, int BM, int BN, int WM, int WN, int S, class Ep>
hipError_t launch_plain(const GemmA& ga, const T* W, int M, int N, int K, const Ep& ep,
                        hipStream_t s, const SplitWs* ws) {
  const int tiles = ((N + BN - 1) / BN) * ((M + BM - 1) / BM);
  constexpr int BK = KCH * 16 / (int)sizeof(T);
  const int nk = K / BK;
  // A grid of one half to one workgroup per CU, or a smaller one whose K is
  // too short to split across workgroups, runs two K groups per workgroup
  // (eight wavefronts, each group half the K steps with its own ring, the
  // halves summed in LDS) when both rings fit the CU's LDS.
  // (The tiles of up to 64 x 64 only: the larger ones run on grids of 256
  // workgroups or more.)
  constexpr bool kFit2 = BM * BN <= 64 * 64 && 2 * S * (BM + BN) * KCH * 16 <= 160 * 1024;
  const bool grid2 = tiles >= kTwoGroupMin ? tiles <= kTwoGroupMax : nk < 24;
  const int kg = kFit2 && grid2 && nk % 2 == 0 && nk >= 8 ? 2 : 1;
  const int nkg = nk / kg;
  int ks = 1;
  // Long-K grids of up to one workgroup per CU split too (in two): at
  // M = 512, K = 3072 that measured 8 % faster, reduction included.
  if (ws && ws->part && tiles < 256 && nkg >= 24) {
    const int cap = kg == 2 ? (tiles < 128 ? 160 : tiles) : (tiles < 128 ? 320 : 2 * tiles);
    for (int c : {16, 12, 8, 6, 4, 3, 2}) {
      if (nkg % c == 0 && nkg / c >= 2 && tiles * c <= cap &&
          (size_t)c * M * N * sizeof(float) <= ws->bytes) {
        ks = c;
        break;
      }
    }
  }
  constexpr int KGI = kFit2 ? 2 : 1;
  if (ks == 1) return launch_tile_kg<T, BM, BN, WM, WN, S, KGI>(kg, ga, W, M, N, K, ep, s, 1);
  const EpPartial pe{ws->part, N, nullptr};
  hipError_t e = launch_tile_kg<T, BM, BN, WM, WN, S, KGI>(kg, ga, W, M, N, K, pe, s, ks);
  if (e != hipSuccess) return e;
  return launch_splitk_reduce(ws->part, ks, M, N, ep, s);
}

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// Steps of at most this many rows run the skinny kernel (16-bit operands).
constexpr int kSkinnyRows = 16;

// Tile choice: the largest tile that still gives about one workgroup per CU.
template <typename T, int MODE, bool NORM, class Ep>
hipError_t dispatch(const GemmA& ga, const T* W, int M, int N, int K, const Ep& ep, hipStream_t s,
                    const SplitWs* ws = nullptr) {
  if (M <= 0 || N <= 0) return hipSuccess;
  if constexpr (sizeof(T) == 2) {
    if (M <= kSkinnyRows && N % 16 == 0 && K % 128 == 0)
      return launch_skinny<T, MODE, NORM>(ga, W, M, N, K, ep, s);
  }
  constexpr int kFill = 256;
  if constexpr (!NORM && MODE == 0) {
    if (cdiv(M, 128) * cdiv(N, 128) >= kFill)
      return launch_plain<T, 128, 128, 2, 4, 2>(ga, W, M, N, K, ep, s, ws);
    if (cdiv(M, 64) * cdiv(N, 128) >= kFill)
      return launch_plain<T, 64, 128, 2, 4, 3>(ga, W, M, N, K, ep, s, ws);
    if (cdiv(M, 64) * cdiv(N, 64) >= kFill * 3 / 4)
      return launch_plain<T, 64, 64, 2, 2, 3>(ga, W, M, N, K, ep, s, ws);
    if (cdiv(M, 32) * cdiv(N, 64) >= kFill * 3 / 4)
      return launch_plain<T, 32, 64, 2, 2, 4>(ga, W, M, N, K, ep, s, ws);
    return launch_plain<T, 32, 32, 2, 2, 4>(ga, W, M, N, K, ep, s, ws);
  } else {
    if (cdiv(M, 128) * cdiv(N, 128) >= kFill)
      return launch_tile<T, 128, 128, 2, 4, 2, MODE, NORM>(ga, W, K, M, N, K, ep, s);
    if (cdiv(M, 64) * cdiv(N, 128) >= kFill)
      return launch_tile<T, 64, 128, 2, 4, 3, MODE, NORM>(ga, W, K, M, N, K, ep, s);
    {
      // three quarters of a workgroup per CU or more in 64 x 96 tiles: two K
      // groups of four wavefronts (both rings: 120 KB of LDS).  At M = 512
      // (QKV 192 tiles, MLP-up 256) +1.2 % on the LM1B-shaped generate; with
      // 128 tiles (MLP-up at M = 256) -2.8 % on the OWT-shaped batch 32.
      const int t96 = cdiv(M, 64) * cdiv(N, 96), nk = K / (KCH * 16 / (int)sizeof(T));
      if (N % 96 == 0 && t96 >= 192 && t96 <= kTwoGroupMax && nk % 2 == 0 && nk >= 8)
        return launch_tile<T, 64, 96, 2, 2, 3, MODE, NORM, 2>(ga, W, K, M, N, K, ep, s);
    }
    // The smaller tiles take two K groups on grids of half to one workgroup
    // per CU as well (the QKV and MLP-up GEMMs at OWT-shaped batch 8 and 16:
    // +1.2 % and +0.4 % on the generate, batch 32 unchanged).
    const int nks = K / (KCH * 16 / (int)sizeof(T));
    auto two = [&](int t) {
      return t >= kTwoGroupMin && t <= kTwoGroupMax && nks % 2 == 0 && nks >= 8;
    };
    if (cdiv(M, 64) * cdiv(N, 64) >= kFill * 3 / 4) {
      if (two(cdiv(M, 64) * cdiv(N, 64)))
        return launch_tile<T, 64, 64, 2, 2, 3, MODE, NORM, 2>(ga, W, K, M, N, K, ep, s);
      return launch_tile<T, 64, 64, 2, 2, 3, MODE, NORM>(ga, W, K, M, N, K, ep, s);
    }
    if (cdiv(M, 32) * cdiv(N, 64) >= kFill * 3 / 4) {
      if (two(cdiv(M, 32) * cdiv(N, 64)))
        return launch_tile<T, 32, 64, 2, 2, 4, MODE, NORM, 2>(ga, W, K, M, N, K, ep, s);
      return launch_tile<T, 32, 64, 2, 2, 4, MODE, NORM>(ga, W, K, M, N, K, ep, s);
    }
    if (two(cdiv(M, 32) * cdiv(N, 32)))
      return launch_tile<T, 32, 32, 2, 2, 4, MODE, NORM, 2>(ga, W, K, M, N, K, ep, s);
    return launch_tile<T, 32, 32, 2, 2, 4, MODE, NORM>(ga, W, K, M, N, K, ep, s);
  }
}

// LayerNorm folding at weight load, one wavefront per output row n:
//   Wout[n][k] = W[n][k] g[k] (rounded to T), c1[n] = sum_k Wout[n][k],
//   c2[n] = sum_k W[n][k] beta[k].
// c1 sums the rounded weights, so the mean term cancels exactly against the
// MFMA products.  Wout may be W itself.
template <typename T>
__global__ void __launch_bounds__(256)
    ln_fold_kernel(const T* W, T* Wout, const float* __restrict__ g,
                   const float* __restrict__ beta, int N, int K, float* c1, float* c2) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (n >= N) return;
  float a = 0.f, b = 0.f;
  for (int k = lane; k < K; k += 64) {
    const float w = to_f(W[(size_t)n * K + k]);
    const T ws = from_f<T>(w * g[k]);
    Wout[(size_t)n * K + k] = ws;
    a += to_f(ws);
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
                     T* out, int ldo, const SplitWs* ws, hipStream_t s) {
  EpBias<T> ep{out, ldo, bias, act == Act::Gelu ? 1 : 0};
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, N, K,
                               ep, s, ws);
}

template <typename T>
hipError_t gemm_f32(const T* A, const T* W, int M, int N, int K, float* out, hipStream_t s) {
  const EpPartial ep{out, N, nullptr};
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, N, K,
                               ep, s, nullptr);
}

template <typename T>
hipError_t gemm_residual(const T* A, const T* W, int M, int N, int K, const float* bias, float* X,
                         T* Xh, float2* lnst, const SplitWs* ws, hipStream_t s) {
  EpResidual<T> ep{X, Xh, N, bias, lnst};
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, N, K,
                               ep, s, ws);
}

template <typename T>
hipError_t gemm_residual_rows(const T* A, bool a_rows, KfStepGeom g, const T* W, int M, int N,
                              int K, const float* bias, float* X, T* Xh, float2* lnst,
                              const SplitWs* ws, hipStream_t s) {
  EpResidual<T, true> ep{X, Xh, N, bias, lnst, g.k, g.R, g.nr};
  if (a_rows)  // A holds every row of the step; GEMM row m reads the same row as it writes
    return dispatch<T, 1, false>(GemmA{A, K, g.B * g.R, nullptr, nullptr, nullptr, g}, W, M, N, K,
                                 ep, s, ws);
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, N, K,
                               ep, s, ws);
}

template <typename T>
hipError_t gemm_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                          const T* pos, const T* temb, float* X, T* Xh, float2* lnst,
                          KfStepGeom g, const KfDevState* st, const SplitWs* ws, hipStream_t s) {
  EpNoiseOut<T> ep{X, Xh, bias, pos, temb, st, g, d, lnst};
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, d, K,
                               ep, s, ws);
}

template <typename T>
hipError_t gemm_qkv_ln(const T* Xh, const LnFold& ln, const T* W, int M, int d, const float* bias,
                       T* Q, T* kv, KfStepGeom g, KfKvGeom kg, int layer, const KfDevState* st,
                       const float2* rope, hipStream_t s) {
  EpQKV<T> ep{Q, kv, bias, st, g, kg, layer, rope};
  return dispatch<T, 0, true>(GemmA{Xh, d, M, ln.c1, ln.c2, ln.lnst, g, ln.rms}, W, M, 3 * d, d, ep, s);
}

template <typename T>
hipError_t gemm_up_ln(const T* Xh, const LnFold& ln, const T* W, int M, int N, int d,
                      const float* bias, T* out, hipStream_t s) {
  EpBias<T> ep{out, N, bias, 1};
  return dispatch<T, 0, true>(GemmA{Xh, d, M, ln.c1, ln.c2, ln.lnst, KfStepGeom{}, ln.rms}, W, M, N, d, ep,
                              s);
}

template <typename T>
hipError_t gemm_up_ln_rows(const T* Xh, const LnFold& ln, KfStepGeom g, const T* W, int M, int N,
                           int d, const float* bias, T* out, hipStream_t s) {
  EpBias<T> ep{out, N, bias, 1};
  return dispatch<T, 1, true>(GemmA{Xh, d, g.B * g.R, ln.c1, ln.c2, ln.lnst, g, ln.rms}, W, M, N, d,
                              ep, s);
}

template <typename T>
hipError_t gemm_head_ln(const T* Xh, const LnFold& ln, const T* W, int M, int Vpad, int V, int d,
                        int gather, KfStepGeom g, float* pval, int* pidx, float* logits,
                        hipStream_t s, KfDevState* commit_st, int commit_nr) {
  if (M <= 0) return hipSuccess;
  EpHead ep{nullptr, pval, pidx, logits, V, Vpad / kHeadTileN, commit_st, g, commit_nr};
  const GemmA ga{Xh, d, g.B * g.R, ln.c1, ln.c2, ln.lnst, g, ln.rms};
  auto go = [&](auto mode) {
    constexpr int MODE = decltype(mode)::value;
    if (M <= 32)
      return launch_tile<T, 32, kHeadTileN, 1, 4, 3, MODE, true>(ga, W, d, M, Vpad, d, ep, s);
    // 128-row tiles from 129 rows on: each weight tile is read by half as many
    // workgroups (LM1B-shaped batch 64, 256 head rows: 24.5 -> 19.3 us per head)
    if (M <= 128)
      return launch_tile<T, 64, kHeadTileN, 2, 4, 3, MODE, true>(ga, W, d, M, Vpad, d, ep, s);
    return launch_tile<T, 128, kHeadTileN, 2, 2, 2, MODE, true>(ga, W, d, M, Vpad, d, ep, s);
  };
  if (gather == 2) return go(std::integral_constant<int, 2>{});
  return go(std::integral_constant<int, 1>{});
}

template <typename T>
hipError_t gemm_qkv_seq(const T* Xh, const LnFold& ln, const T* W, int M, int d, const float* bias,
                        T* Q, T* K, T* V, int n, int ldk, int koff, int H, int N, int k, int round,
                        const float2* rope, hipStream_t s) {
  EpQKVSeq<T> ep{Q, K, V, bias, n, ldk, koff, H, d / H, N, k, round, rope};
  return dispatch<T, 0, true>(GemmA{Xh, d, M, ln.c1, ln.c2, ln.lnst, KfStepGeom{}, ln.rms}, W, M, 3 * d, d,
                              ep, s);
}

template <typename T>
hipError_t gemm_seq_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                              const T* pos, const T* temb, float* X, T* Xh, float2* lnst, int n,
                              int off, int N, int k, int shift, const SplitWs* ws, hipStream_t s) {
  EpSeqNoise<T> ep{X, Xh, bias, pos, temb, n, off, N, k, shift, d, lnst};
  return dispatch<T, 0, false>(GemmA{A, K, M, nullptr, nullptr, nullptr, KfStepGeom{}}, W, M, d, K,
                               ep, s, ws);
}

template <typename T>
hipError_t gemm_head_sample(const T* Xh, const LnFold& ln, const T* W, int M, int Vpad, int V, int d,
                            int row0, int rows_per_seq, const float* tau, float* pmax, float* psub,
                            float* logits, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  EpHeadSample ep{nullptr, pmax, psub, logits, tau, row0, rows_per_seq, V, Vpad / kHeadTileN};
  const GemmA ga{Xh + (size_t)row0 * d, d, M, ln.c1, ln.c2, ln.lnst + (size_t)row0 * (d / 16),
                 KfStepGeom{}, ln.rms};
  if (M <= 32)
    return launch_tile<T, 32, kHeadTileN, 1, 4, 3, 0, true>(ga, W, d, M, Vpad, d, ep, s);
  if (M <= 512)
    return launch_tile<T, 64, kHeadTileN, 2, 4, 3, 0, true>(ga, W, d, M, Vpad, d, ep, s);
  return launch_tile<T, 128, kHeadTileN, 2, 2, 2, 0, true>(ga, W, d, M, Vpad, d, ep, s);
}

template <typename T>
hipError_t launch_ln_fold(const T* W, T* Wout, const float* g, const float* beta, int N, int K,
                          float* c1, float* c2, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  launch(ln_fold_kernel<T>, dim3((N + 3) / 4), dim3(256), 0, s, W, Wout, g, beta, N, K,
                     c1, c2);
  return hipGetLastError();
}

#define KF_INST(T)                                                                                 \
  template hipError_t gemm_f32<T>(const T*, const T*, int, int, int, float*, hipStream_t);          \
  template hipError_t gemm_bias<T>(const T*, const T*, int, int, int, const float*, Act, T*, int, \
                                   const SplitWs*, hipStream_t);                                   \
  template hipError_t gemm_residual<T>(const T*, const T*, int, int, int, const float*, float*,   \
                                       T*, float2*, const SplitWs*, hipStream_t);                  \
  template hipError_t gemm_noise_out<T>(const T*, const T*, int, int, int, const float*,          \
                                        const T*, const T*, float*, T*, float2*, KfStepGeom,       \
                                        const KfDevState*, const SplitWs*, hipStream_t);           \
  template hipError_t gemm_qkv_ln<T>(const T*, const LnFold&, const T*, int, int, const float*,   \
                                     T*, T*, KfStepGeom, KfKvGeom, int, const KfDevState*,         \
                                     const float2*, hipStream_t);                                  \
  template hipError_t gemm_up_ln<T>(const T*, const LnFold&, const T*, int, int, int,             \
                                    const float*, T*, hipStream_t);                                \
  template hipError_t gemm_up_ln_rows<T>(const T*, const LnFold&, KfStepGeom, const T*, int, int,  \
                                         int, const float*, T*, hipStream_t);                      \
  template hipError_t gemm_residual_rows<T>(const T*, bool, KfStepGeom, const T*, int, int, int,   \
                                            const float*, float*, T*, float2*, const SplitWs*,     \
                                            hipStream_t);                                          \
  template hipError_t gemm_head_ln<T>(const T*, const LnFold&, const T*, int, int, int, int, int, \
                                      KfStepGeom, float*, int*, float*, hipStream_t, KfDevState*,  \
                                      int);                                                        \
  template hipError_t gemm_qkv_seq<T>(const T*, const LnFold&, const T*, int, int, const float*,  \
                                      T*, T*, T*, int, int, int, int, int, int, int,               \
                                      const float2*, hipStream_t);                                 \
  template hipError_t gemm_seq_noise_out<T>(const T*, const T*, int, int, int, const float*,      \
                                            const T*, const T*, float*, T*, float2*, int, int, int, \
                                            int, int, const SplitWs*, hipStream_t);                \
  template hipError_t gemm_head_sample<T>(const T*, const LnFold&, const T*, int, int, int, int,  \
                                          int, int, const float*, float*, float*, float*,          \
                                          hipStream_t);                                            \
  template hipError_t launch_ln_fold<T>(const T*, T*, const float*, const float*, int, int,       \
                                        float*, float*, hipStream_t);
KF_INST(float)
KF_INST(bf16)
#undef KF_INST

}  // namespace kf
