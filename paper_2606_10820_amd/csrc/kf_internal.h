// kf_internal.h -- internal declarations shared by the library's HIP sources.
// Not part of the public ABI (include/kforcing.h is).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

typedef __bf16 bf16;

// Device-resident sequence state.  Kernels read the committed context length
// C from here (never from a launch argument) so that a step's launches are
// identical from one step to the next.
// LayerNorm statistics of the residual stream, written by every kernel that
// writes residual rows: per 16-column group of a row, (s, m2) = (the sum of
// its 16 values, the sum of their squared deviations from the group mean
// s / 16).  Consumers merge the groups of a row with the pairwise update of
// Chan, Golub and LeVeque for equal counts: mean mu = (sum of s) / K and
// K var = sum of (m2 + (s - 16 mu)^2 / 16), which has no E[x^2] - mu^2
// cancellation when |mu| is large against the spread; with mu = 0 the same sum
// is the row's sum of squares (RMSNorm).
__host__ __device__ inline float ln_group_sq(float2 st, float mu) {
  const float t = st.x - 16.0f * mu;
  return st.y + t * t * (1.0f / 16.0f);
}
// (s, m2) of 16 values held 8 by this lane and 8 by lane ^ 1 (both lanes call).
__device__ inline float2 ln_group16(const float (&v)[8]) {
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) a += v[i];
  a += __shfl_xor(a, 1, 64);
  const float mean = a * (1.0f / 16.0f);
  float m2 = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float t = v[i] - mean;
    m2 += t * t;
  }
  m2 += __shfl_xor(m2, 1, 64);
  return make_float2(a, m2);
}
// (s, m2) of 16 values held by one thread.
__device__ inline float2 ln_group16_one(const float (&v)[16]) {
  float a = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) a += v[i];
  const float mean = a * (1.0f / 16.0f);
  float m2 = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float t = v[i] - mean;
    m2 += t * t;
  }
  return make_float2(a, m2);
}

struct KfDevState {
  int C;    // committed context length (positions 0..C-1 hold real-token K/V)
  int err;  // bit 0: a token id outside [0, V) was replaced by 0; bit 1: a bad temperature
  int pad[14];
};

// Where a step writes the tokens it selects.
struct KfOutDesc {
  int32_t* out;    // destination
  int stride;      // per-sequence stride of out (elements)
  int gen_base;    // >= 0: generation run, element index = emitted position - gen_base
                   // <  0: element index = head row index within the sequence
  int32_t* pend;   // pending-token buffer [slots][pend_stride] for the next step
  int pend_stride;
};

// Geometry of one step: B sequences, R = nr + k rows each (nr real rows, then
// k noise rows), row (b, i) stored at index b * R + i.
//
// Lock-step batches (map == null): step sequence b is sequence slot b and every
// sequence has the committed length KfDevState::C.  Continuous batching
// (map != null): step sequence b is slot map[b], whose committed length is
// cs[map[b]]; the slot picks its KV pages, pending tokens and temperature.
struct KfStepGeom {
  int B, R, nr, k;
  const int* map = nullptr;  // [B] sequence slots of the step, or null
  int* cs = nullptr;         // [slots] committed lengths (with map), or null
  int qoff = 0;              // first row of each sequence the attention computes
  __device__ inline int slot(int b) const { return map ? map[b] : b; }
  __device__ inline int ctx(const KfDevState* st, int b) const { return map ? cs[map[b]] : st->C; }
};

// Geometry of the KV cache, in pages of kPage = 128 slots of one sequence.  A
// page holds every layer: [L][2][H][128 * dh] elements, per head the keys
// [128][dh] (slot-major) and the values transposed in blocks of kVBlk = 4
// slots, [32][dh][4]: the 4 slots of a block are contiguous for each value
// row, and consecutive value rows of a block are adjacent, so the rows a step
// appends (positions advance by whole blocks) are written as lane-contiguous
// runs; 8 consecutive slots of a value row (one P.V operand fragment) are two
// 4-slot pieces.  Slot s of sequence slot q lives in page
// ptab[q * (T / 128) + s / 128]; without a page table (lock-step batches)
// sequence q owns pages q * (T / 128) onwards.  T is the per-sequence capacity
// rounded up to a whole page.  (Pages of 128 rather than 64 slots measured
// faster in the QKV epilogue's KV append.)
constexpr int kPage = 128;
constexpr int kVBlk = 4;
struct KfKvGeom {
  int L, H, T, dh;
  const int* ptab = nullptr;  // [slots][T / kPage] page ids, or null
  __host__ __device__ unsigned page_elems() const { return (unsigned)(L * 2 * H * kPage * dh); }
  // Offset of (layer, K or V, head) within a page (a page has < 2^31 elements).
  __host__ __device__ unsigned head_off(int layer, int which, int h) const {
    return (unsigned)(((layer * 2 + which) * H + h) * (kPage * dh));
  }
  // Offset of value (slot s, row e) within a head's value blocks.
  __host__ __device__ static unsigned vt_off(int s, int e, int dh) {
    return (unsigned)(((s % kPage) / kVBlk) * (dh * kVBlk) + e * kVBlk + (s % kVBlk));
  }
  // First element of the page holding slot s of sequence slot q.
  __device__ inline size_t page_base(int q, int s) const {
    const unsigned np = (unsigned)T / kPage, j = (unsigned)s / kPage;
    const unsigned pg = ptab ? (unsigned)ptab[q * np + j] : q * np + j;
    return (size_t)pg * page_elems();
  }
};

// ------------------------------------------------------------------ Philox
// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32 -> 64-bit
// multiplies with a Weyl key schedule.  Noise for sequence b at emitted
// position p: counter (p, b, 2, 0), key (seed lo, seed hi), u = (w0 >> 8) 2^-24.
__host__ __device__ inline void kf_philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    uint32_t n3 = (uint32_t)p0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
  }
}

__host__ __device__ inline float kf_noise_u(uint64_t seed, int b, int p) {
  uint32_t c[4] = {(uint32_t)p, (uint32_t)b, 2u, 0u};
  kf_philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  return (float)(c[0] >> 8) * (1.0f / 16777216.0f);
}

// ------------------------------------------------------------ launchers
// All return hipGetLastError() of their launch (hipSuccess when nothing ran).
namespace kf {

// Kernel timing.  While a kernel class is being timed the host points
// launch_timer at an event pair: the first kernel of the launcher records
// `start` on its own dispatch and every kernel records `stop`, so the interval
// is exactly the launcher's kernels (no event packets between them).
struct LaunchTimer {
  hipEvent_t start, stop;
  bool started;
};
extern thread_local LaunchTimer* launch_timer;

template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  if (LaunchTimer* t = launch_timer) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, t->started ? nullptr : t->start, t->stop,
                          0u, args...);
    t->started = true;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
  }
}

enum class Act { None = 0, Gelu = 1 };

// fp32 workspace of the split-K GEMMs (plain GEMMs whose grids cannot fill the
// chip run as K splits into it, then a reduction); null part: no split.
struct SplitWs {
  float* part;
  size_t bytes;
};

// The noise encoder's output computed ahead for whole chunks of the passes of a
// lock-step generate (the encoder depends on u, the position and the
// temperature only, never on the emitted tokens).  nz [qp passes][B*k][d]
// (fp32, without the second layer's bias): pass p's rows sit in chunk slot
// p % qp.  pass >= 0 names the step's pass; pass < 0 derives it from the
// committed length, pass = (C - N) / k + 1 (a decode block of the generate).
struct NoiseAhead {
  const float* nz;
  const float* bias;  // second noise-MLP layer's bias [d]
  const void* temb;   // per-slot temperature embedding [slots][d] (compute dtype), or null
  int N;              // prompt length of the generate
  int qp;             // passes per chunk
  int pass;
};

// Real-row embedding: X[b*R + i] = tok[toks[q*tok_stride + i]] + pos[C_b + i], i < nr,
// with its compute-dtype copy Xh and LayerNorm partial sums lnst (see gemm_residual);
// q = b, or the step's sequence slot when toks_by_slot (the pending-token buffer).
// With na, also the step's k noise rows from the encoder output computed ahead:
// X[b*R + nr + j] = (nz + bias) + pos[C_b + nr + j] (+ temb[slot b]).
template <typename T>
hipError_t launch_embed_real(float* X, T* Xh, float2* lnst, const T* tok, const T* pos,
                             const int32_t* toks, int tok_stride, int toks_by_slot, KfStepGeom g,
                             int d, int V, KfDevState* st, hipStream_t s,
                             const NoiseAhead* na = nullptr);

// Sinusoids of the noise rows of passes pass0 .. pass0 + npass - 1 of a
// lock-step generate (prompt length N, sequence b in slot b) into
// S [npass*B*k][d]: row ((pass - pass0) B + b) k + j has u from the device
// Philox stream at position N + pass k + j.
template <typename T>
hipError_t launch_noise_sinusoid_ahead(T* S, uint64_t seed, const double* omega, int B, int k,
                                       int N, int pass0, int npass, int d, hipStream_t s);

// Sinusoid of each noise row's u into S [B*k][d]; u from noise [B*k] or, when
// noise is null, from the device Philox stream at positions C_b + nr + j.
// The u actually used are written to u_out [B*k] when it is not null.
template <typename T>
hipError_t launch_noise_sinusoid(T* S, const float* noise, uint64_t seed, const double* omega,
                                 KfStepGeom g, int d, const KfDevState* st, float* u_out,
                                 hipStream_t s);

// Key-split workspace of the attention: per (sequence, head, query row, split)
// entry the running max m, the sum l and the unnormalised output o[d_head]
// (fp32).  ns is chosen by the launcher (1 = no split).
struct AttnSplit {
  float* m;
  float* l;
  float* o;
  int entries;  // capacity in entries
  int ns;
};
// Block attention over the KV cache for every (sequence, head, query block).
template <typename T>
hipError_t launch_attention(const T* Q, const T* kv, T* O, const KfDevState* st, KfStepGeom g,
                            KfKvGeom kg, int layer, const AttnSplit& ws, hipStream_t s);

// GEMM family: C = epilogue(A[M][K] . W[N][K]^T), fp32 accumulation.
template <typename T>
hipError_t gemm_bias(const T* A, const T* W, int M, int N, int K, const float* bias, Act act,
                     T* out, int ldo, const SplitWs* ws, hipStream_t s);
// out[M][N] = A . W^T in fp32 (no bias, no split).
template <typename T>
hipError_t gemm_f32(const T* A, const T* W, int M, int N, int K, float* out, hipStream_t s);
// Residual update X[M][N] += C + bias; with a 16-bit T the updated rows are
// also written to Xh (the compute-dtype copy of the residual stream; for fp32,
// Xh aliases X and is not written).  Every writer of the residual stream also
// writes lnst [rows][N / 16]: per 16 columns of the updated row, the sum and
// the sum of squared deviations from their mean, the input of the next folded
// LayerNorm.
template <typename T>
hipError_t gemm_residual(const T* A, const T* W, int M, int N, int K, const float* bias, float* X,
                         T* Xh, float2* lnst, const SplitWs* ws, hipStream_t s);
// The same for the head rows of a step only (the last layer of a step with
// noise rows, whose real rows feed nothing after their K/V append): M = B k
// GEMM rows, row m updating stream row (m / k) R + nr + m % k of g.  With
// a_rows, A holds every row of the step and GEMM row m reads that same row
// (the attention output); otherwise A has the M rows (the MLP hidden layer).
template <typename T>
hipError_t gemm_residual_rows(const T* A, bool a_rows, KfStepGeom g, const T* W, int M, int N,
                              int K, const float* bias, float* X, T* Xh, float2* lnst,
                              const SplitWs* ws, hipStream_t s);
// LayerNorm folded into a GEMM whose weights were scaled by the gain at load
// (W' = W diag(gain)): c1 = W' 1 and c2 = W shift.  A rows come from the
// compute-dtype residual copy Xh [rows][d]; each row's mean and variance come
// from its partial sums in lnst.
struct LnFold {
  const float* c1;
  const float* c2;
  const float2* lnst;  // partial row sums of the residual stream (see gemm_residual)
  int rms;             // RMSNorm: no mean (mu = 0, rstd from the mean square)
};
// rope (optional): rotary table [n_ctx][d_rot/2] (cos, sin) with d_rot =
// min(64, d_head); when set, Q and K are rotated at each row's position C + i.
template <typename T>
hipError_t gemm_qkv_ln(const T* Xh, const LnFold& ln, const T* W, int M, int d, const float* bias,
                       T* Q, T* kv, KfStepGeom g, KfKvGeom kg, int layer, const KfDevState* st,
                       const float2* rope, hipStream_t s);
template <typename T>
hipError_t gemm_up_ln(const T* Xh, const LnFold& ln, const T* W, int M, int N, int d,
                      const float* bias, T* out, hipStream_t s);
// MLP-up of the head rows of a step only (see gemm_residual_rows): A row m is
// stream row (m / k) R + nr + m % k, the M = B k output rows are contiguous.
template <typename T>
hipError_t gemm_up_ln_rows(const T* Xh, const LnFold& ln, KfStepGeom g, const T* W, int M, int N,
                           int d, const float* bias, T* out, hipStream_t s);
template <typename T>
hipError_t gemm_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                          const T* pos, const T* temb, float* X, T* Xh, float2* lnst,
                          KfStepGeom g, const KfDevState* st, const SplitWs* ws, hipStream_t s);
// Head over the final LayerNorm of the selected rows (gather: 1 = noise rows
// of the step, 2 = last real row per sequence): per (row, 128-column tile) the
// maximum and its lowest column index into pval/pidx [M][Vpad/128]; columns
// >= V are excluded.  When logits is not null the fp32 logits [M][V] are
// written as well.  W is the gain-scaled token table [Vpad][d].  With
// commit_st, the head also commits the step (C += commit_nr, or per slot
// through g's slot map) once its first workgroup is done: nothing after the
// layers reads C but the selection, which is then told commit_nr.
template <typename T>
hipError_t gemm_head_ln(const T* Xh, const LnFold& ln, const T* W, int M, int Vpad, int V, int d,
                        int gather, KfStepGeom g, float* pval, int* pidx, float* logits,
                        hipStream_t s, KfDevState* commit_st = nullptr, int commit_nr = 0);
// Head of a temperature-scaled sampling pass (teacher targets) over rows
// row0 .. row0 + M - 1 of the step (all rows are real rows; row r belongs to
// sequence r / rows_per_seq, temperature tau[r / rows_per_seq]): per launch
// row m and 128-column tile t, pmax [M][n_tiles] = max over columns < V of
// l / tau and psub [M][n_tiles][8] = per 16-column group, sum exp(l / tau -
// pmax).  When logits is not null the fp32 logits [M][V] are written too.
template <typename T>
hipError_t gemm_head_sample(const T* Xh, const LnFold& ln, const T* W, int M, int Vpad, int V, int d,
                            int row0, int rows_per_seq, const float* tau, float* pmax, float* psub,
                            float* logits, hipStream_t s);
// Inverse-CDF selection from the sampling head's partials: for launch row m
// (step row row0 + m, sequence b = (row0 + m) / rows_per_seq) the smallest
// column j with F_j > u[row0 + m], F the CDF of softmax(l / tau_b); the
// crossing group's 16 logits are recomputed from Xh, the LayerNorm partial
// sums and the head weights.  A tau outside (0, inf) sets error bit 1 and
// selects 0.  Writes targets[row0 + m].
template <typename T>
hipError_t launch_teacher_select(const float* pmax, const float* psub, int n_tiles, int V,
                                 const T* Xh, const float2* lnst, const T* W, const float* c1,
                                 const float* c2, int rms, int d, const float* tau, const float* u,
                                 int row0, int M, int rows_per_seq, int32_t* targets, KfDevState* st,
                                 hipStream_t s);

// Whole-sequence forward of the teacher rollout (SingleForward / DoubleForward
// passes).  Rows of sequence b are residual rows b*n .. b*n + n - 1.
//   gemm_qkv_seq: LayerNorm-folded QKV; Q to [B][H][n][dh], K and V to
//     [B][H][ldk][dh] at keys koff + i.
//   gemm_seq_noise_out: second noise-MLP layer; noise row (b, t, j) of N groups
//     of k to residual row b*n + off + t*k + j, position t + shift + j.
//   launch_embed_group: token rows (b, t, j) likewise, tokens [B][N*k].
// With rope set, Q and K rows are rotated at their positions in the round's
// layout (round 1: context i, then noise (t, j) at t + 1 + j; round 2:
// Future-1 (t, j) at t + 1 + j, then Future-2 at t + 1 + k + j).
template <typename T>
hipError_t gemm_qkv_seq(const T* Xh, const LnFold& ln, const T* W, int M, int d, const float* bias,
                        T* Q, T* K, T* V, int n, int ldk, int koff, int H, int N, int k, int round,
                        const float2* rope, hipStream_t s);
template <typename T>
hipError_t gemm_seq_noise_out(const T* A, const T* W, int M, int d, int K, const float* bias,
                              const T* pos, const T* temb, float* X, T* Xh, float2* lnst, int n,
                              int off, int N, int k, int shift, const SplitWs* ws, hipStream_t s);
template <typename T>
hipError_t launch_embed_group(float* X, T* Xh, float2* lnst, const T* tok, const T* pos,
                              const int32_t* toks, int B, int N, int k, int n, int off, int shift,
                              int d, int V, KfDevState* st, hipStream_t s);

// Fold a LayerNorm into the GEMM that consumes it: Wout = W diag(gain) in T,
// c1 = Wout 1, c2 = W shift; W [N][K], Wout may alias W.
template <typename T>
hipError_t launch_ln_fold(const T* W, T* Wout, const float* gain, const float* shift, int N, int K,
                          float* c1, float* c2, hipStream_t s);
constexpr int kHeadTileN = 128;

// Argmax over the head partials of each row, ties to the lowest id; writes the
// selected tokens per KfOutDesc.  rows = B * k.  committed: what the head has
// already added to C (the context length of the step is C - committed).
hipError_t launch_argmax_select(const float* pval, const int* pidx, int n_tiles, KfStepGeom g,
                                const KfDevState* st, KfOutDesc od, hipStream_t s,
                                int committed = 0);

// Inverse-CDF sampling of one token per sequence from fp32 logits [B][V]:
// smallest m with F_m > u.  u from u_in [B] or, when null, the Philox stream
// at position C + nr.
hipError_t launch_icdf_select(const float* logits, int V, const float* u_in, uint64_t seed,
                              KfStepGeom g, const KfDevState* st, KfOutDesc od, hipStream_t s);

// C += nr (end of step): KfDevState::C, or with g.map the committed length of
// each of the step's sequence slots.
hipError_t launch_commit(KfDevState* st, KfStepGeom g, int nr, hipStream_t s);
// Committed length 0 for each of the step's sequence slots (g.map required).
hipError_t launch_seq_reset(KfStepGeom g, hipStream_t s);

// Small host-to-device updates carried in the launch arguments (copied at
// launch, so the host may reuse its arrays at once): dst[idx[i]] = val[i].
constexpr int kScatterMax = 240;
struct KfScatter {
  int n;
  int idx[kScatterMax];
  int val[kScatterMax];
};
hipError_t launch_scatter_i32(int* dst, const KfScatter& u, hipStream_t s);

// Device Philox noise for n positions starting at p0, [B][n].
hipError_t launch_fill_noise(float* out, uint64_t seed, int B, int p0, int n, hipStream_t s);

// fp32 -> T conversion of n elements; zero fill of n elements of T.
template <typename T>
hipError_t launch_convert(const float* src, T* dst, size_t n, hipStream_t s);
template <typename T>
hipError_t launch_zero(T* dst, size_t n, hipStream_t s);
hipError_t launch_copy_f32(const float* src, float* dst, size_t n, hipStream_t s);
hipError_t launch_zero_i32(int* dst, size_t n, hipStream_t s);

// Attention under a training mask (KF_MASK_SINGLE / KF_MASK_DOUBLE of
// include/kforcing.h): Q [B*H][rows][dh], K, V [B*H][keys][dh], O like Q, bf16;
// dh in {32, 64, 128}.  rows and keys as given by the two helpers.
int training_attention_rows(int mask, int N, int k);
int training_attention_keys(int mask, int N, int k);
hipError_t launch_training_attention(int mask, int B, int H, int N, int k, int dh, const bf16* Q,
                                     const bf16* K, const bf16* V, bf16* O, float scale,
                                     hipStream_t s);
// The same with K, V holding ldk keys per head and O written as the rows of a
// residual stream, [B][rows][H][dh].
hipError_t launch_training_attention_seq(int mask, int B, int H, int N, int k, int dh, const bf16* Q,
                                         const bf16* K, const bf16* V, int ldk, bf16* O,
                                         float scale, hipStream_t s);

}  // namespace kf
