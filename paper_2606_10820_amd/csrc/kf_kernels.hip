// kf_kernels.hip -- gfx950 kernels of the K-Forcing decode step other than the
// GEMM family: real-row embedding, noise sinusoid, block attention,
// token selection (argmax / inverse CDF) and small utilities.
#include <float.h>
#include <math.h>

#include "kf_internal.h"
#include "kf_attn.h"

namespace kf {

namespace {

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(bf16 x) { return (float)x; }
template <typename T>
__device__ inline T from_f(float x);
template <>
__device__ inline float from_f<float>(float x) { return x; }
template <>
__device__ inline bf16 from_f<bf16>(float x) { return (bf16)x; }

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// ------------------------------------------------------------ embedding
// Real rows (Appendix C.1, Embed): token table row plus learned position.
// With nz (the noise encoder's output for whole chunks of passes, computed
// ahead by kf_generate: NoiseAhead), workgroups past the real rows write the
// step's noise rows from it: noise MLP output + its bias + position (+ the
// sequence's temperature embedding), the sums taken in the order the noise
// GEMM's epilogue takes them.
template <typename T>
__global__ void __launch_bounds__(256)
    embed_real_kernel(float* __restrict__ X, T* __restrict__ Xh, float2* __restrict__ lnst,
                      const T* __restrict__ tok, const T* __restrict__ pos,
                      const int32_t* __restrict__ toks, int tok_stride, int toks_by_slot,
                      KfStepGeom g, int d, int V, KfDevState* st, NoiseAhead na) {
  const int grp = threadIdx.x;  // one thread per 16 columns (d <= 2048)
  if ((int)blockIdx.x >= g.B * g.nr) {
    const int q = blockIdx.x - g.B * g.nr, b = q / g.k, j = q - b * g.k;
    const int C = g.ctx(st, b);
    int pass = na.pass >= 0 ? na.pass : (C - na.N) / g.k + 1;
    pass = pass > 0 ? pass : 0;  // (a lock-step generate has C >= N here)
    const size_t row = (size_t)b * g.R + g.nr + j;
    const float* nzr = na.nz + ((size_t)(pass % na.qp) * g.B * g.k + q) * d;
    const T* pe = pos + (size_t)(C + g.nr + j) * d;
    const T* tb = na.temb ? static_cast<const T*>(na.temb) + (size_t)g.slot(b) * d : nullptr;
    if (grp < d / 16) {
      float v[16];
#pragma unroll
      for (int c = 0; c < 16; ++c) {
        const int e = grp * 16 + c;
        v[c] = (nzr[e] + na.bias[e]) + to_f(pe[e]);
        if (tb) v[c] += to_f(tb[e]);
        X[row * d + e] = v[c];
        if constexpr (sizeof(T) == 2) Xh[row * d + e] = from_f<T>(v[c]);
      }
      lnst[row * (d / 16) + grp] = ln_group16_one(v);
    }
    return;
  }
  const int r = blockIdx.x;
  const int b = r / g.nr, i = r % g.nr;
  const int C = g.ctx(st, b);
  int t = toks[(size_t)(toks_by_slot ? g.slot(b) : b) * tok_stride + i];
  if (t < 0 || t >= V) {
    if (threadIdx.x == 0) atomicOr(&st->err, 1);
    t = 0;
  }
  const size_t row = (size_t)b * g.R + i;
  float* x = X + row * d;
  const T* te = tok + (size_t)t * d;
  const T* pe = pos + (size_t)(C + i) * d;
  T* xh = Xh + row * d;
  // the row and its LayerNorm partials
  if (grp < d / 16) {
    float v[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int e = grp * 16 + c;
      v[c] = to_f(te[e]) + to_f(pe[e]);
      x[e] = v[c];
      if constexpr (sizeof(T) == 2) xh[e] = from_f<T>(v[c]);
    }
    lnst[row * (d / 16) + grp] = ln_group16_one(v);
  }
}

// ------------------------------------------------------- noise sinusoid
// One row of the sinusoid of u (the expansion described below).
template <typename T>
__device__ inline void sinusoid_row(T* __restrict__ row, float u, const double* __restrict__ omega,
                                    int d) {
  const int h = d / 2;
  const double su = 1000.0 * (double)u;
  for (int i = threadIdx.x; i < h; i += blockDim.x) {
    double a = su * omega[i];
    double sn, cs;
    sincos(a, &sn, &cs);
    row[i] = from_f<T>((float)cs);
    row[h + i] = from_f<T>((float)sn);
  }
}

// Noise rows: the scalar u of each noise token is expanded into d features,
// cos(a_i) then sin(a_i) with a_i = 1000 u omega_i, omega_i = 10000^(-i/(d/2)),
// evaluated in double so that fp32 u keeps its full resolution.
template <typename T>
__global__ void __launch_bounds__(256)
    noise_sinusoid_kernel(T* __restrict__ S, const float* __restrict__ noise, uint64_t seed,
                          const double* __restrict__ omega, KfStepGeom g, int d,
                          const KfDevState* st, float* __restrict__ u_out) {
  const int m = blockIdx.x;
  const int b = m / g.k, j = m % g.k;
  float u = noise ? noise[m] : kf_noise_u(seed, g.slot(b), g.ctx(st, b) + g.nr + j);
  if (u_out && threadIdx.x == 0) u_out[m] = u;
  sinusoid_row(S + (size_t)m * d, u, omega, d);
}

// The sinusoids of the noise rows of passes pass0, pass0 + 1, ... of a
// lock-step generate (sequence b in slot b, prompt length N, k rows a pass):
// row m = ((pass - pass0) B + b) k + j holds u at position N + pass k + j.
template <typename T>
__global__ void __launch_bounds__(256)
    noise_sinusoid_ahead_kernel(T* __restrict__ S, uint64_t seed, const double* __restrict__ omega,
                                int B, int k, int N, int pass0, int d) {
  const int m = blockIdx.x, bk = B * k;
  const int pass = pass0 + m / bk, q = m % bk, b = q / k, j = q - b * k;
  sinusoid_row(S + (size_t)m * d, kf_noise_u(seed, b, N + pass * k + j), omega, d);
}

// ------------------------------------------------------ block attention
// One workgroup per (sequence, head, block of 16 query rows).  The query rows
// of a step sit at cache slots C + i (real rows first, then noise rows) and
// attend causally over slots [0, C + i]: real row i sees the context and real
// rows <= i, noise row j sees the context, every real row and noise rows <= j
// (the fully causal layout of Sec. 3.3; mask of the decode window, App. C).
// Online softmax over 64-key tiles streamed from the per-sequence cache.
template <typename T, int DH>
__global__ void __launch_bounds__(256)
    attention_kernel(const T* __restrict__ Q, const T* __restrict__ kv, T* __restrict__ O,
                     const KfDevState* st, KfStepGeom g, KfKvGeom kg, int layer, float scale) {
  constexpr int QB = 16, KT = 64, EPT = DH / 16;
  const int H = kg.H, d = H * DH;
  const int b = blockIdx.x / H, h = blockIdx.x % H;
  const int q0 = g.qoff + blockIdx.y * QB;
  const int nq = min(QB, g.R - q0);
  const int C = g.ctx(st, b), seq = g.slot(b);
  const int nkeys = C + q0 + nq;

  __shared__ float sQ[QB][DH];
  __shared__ float sK[KT][DH + 1];
  __shared__ float sV[KT][DH];
  __shared__ float sP[QB][KT];

  const int tid = threadIdx.x;
  for (int idx = tid; idx < QB * DH; idx += 256) {
    int qi = idx / DH, e = idx % DH;
    sQ[qi][e] = (qi < nq) ? to_f(Q[((size_t)b * g.R + q0 + qi) * d + h * DH + e]) * scale : 0.f;
  }
  const int qi = tid >> 4, r16 = tid & 15;
  const int qslot = C + q0 + qi;
  float m_run = -INFINITY, l_run = 0.f;
  float o[EPT];
#pragma unroll
  for (int c = 0; c < EPT; ++c) o[c] = 0.f;

  static_assert(kPage % KT == 0, "a key tile lies in one KV page");
  for (int kt0 = 0; kt0 < nkeys; kt0 += KT) {
    const T* page = kv + kg.page_base(seq, kt0);
    const T* Kb = page + kg.head_off(layer, 0, h);
    const T* Vb = page + kg.head_off(layer, 1, h);
    const int p0 = kt0 % kPage;
    __syncthreads();
    for (int idx = tid; idx < KT * DH; idx += 256) {
      int kk = idx / DH, e = idx % DH, slot = kt0 + kk;
      float kx = 0.f, vx = 0.f;
      if (slot < nkeys) {
        kx = to_f(Kb[(size_t)(p0 + kk) * DH + e]);
        vx = to_f(Vb[KfKvGeom::vt_off(p0 + kk, e, DH)]);
      }
      sK[kk][e] = kx;
      sV[kk][e] = vx;
    }
    __syncthreads();
    float sc[4];
    float tmax = -INFINITY;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      int key = r16 * 4 + c, slot = kt0 + key;
      float dot = 0.f;
#pragma unroll 16
      for (int e = 0; e < DH; ++e) dot += sQ[qi][e] * sK[key][e];
      sc[c] = (qi < nq && slot <= qslot) ? dot : -INFINITY;
      tmax = fmaxf(tmax, sc[c]);
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) tmax = fmaxf(tmax, __shfl_xor(tmax, off, 16));
    const float m_new = fmaxf(m_run, tmax);
    const float ref = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __expf(m_run - ref);
    float psum = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float p = __expf(sc[c] - ref);
      sP[qi][r16 * 4 + c] = p;
      psum += p;
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) psum += __shfl_xor(psum, off, 16);
    l_run = l_run * alpha + psum;
    m_run = m_new;
    __syncthreads();
#pragma unroll
    for (int c = 0; c < EPT; ++c) {
      int e = c * 16 + r16;
      float acc = o[c] * alpha;
#pragma unroll 16
      for (int key = 0; key < KT; ++key) acc += sP[qi][key] * sV[key][e];
      o[c] = acc;
    }
  }
  if (qi < nq) {
    T* orow = O + ((size_t)b * g.R + q0 + qi) * d + h * DH;
    const float inv = 1.0f / l_run;
#pragma unroll
    for (int c = 0; c < EPT; ++c) orow[c * 16 + r16] = from_f<T>(o[c] * inv);
  }
}

// Block attention on MFMA (bf16): one workgroup per (sequence, head, block of
// 16 query rows, key split), the block computed by attention_block (kf_attn.h).
// PT selects where the KV pages come from (attention_tiles); each mode is its
// own kernel, so the lock-step one carries no page-table registers.  Up to
// d_head 64 the kernel is held to three wavefronts per SIMD (at most 168
// registers, no spill): the double-buffered K and V fragments would otherwise
// take it to two, and at large batch the KV stream needs the occupancy.
template <int DH, int NW, int PT>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(DH <= 64 ? 3 : 1)))
    attention_mfma_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ kv,
                          bf16* __restrict__ O, const KfDevState* st, KfStepGeom g, KfKvGeom kg,
                          int layer, float scale, AttnSplit sp) {
  const int nqb = (g.R - g.qoff + 15) / 16;
  const int split = blockIdx.x % sp.ns, rest = blockIdx.x / sp.ns;
  const int qb = rest % nqb, bh = rest / nqb;
  attention_block<DH, NW, PT>(Q, kv, O, st, g, kg, layer, scale, sp, bh / kg.H, bh % kg.H, qb,
                              split);
}

template <int DH, int NW>
void launch_attention_mfma(dim3 grid, hipStream_t s, const bf16* Q, const bf16* kv, bf16* O,
                           const KfDevState* st, const KfStepGeom& g, const KfKvGeom& kg, int layer,
                           float scale, const AttnSplit& sp) {
  const dim3 block(64 * NW);
  if (!kg.ptab)
    launch((attention_mfma_kernel<DH, NW, 0>), grid, block, 0, s, Q, kv, O, st, g, kg, layer,
           scale, sp);
  else if (kg.T <= 64 * kPage)
    launch((attention_mfma_kernel<DH, NW, 1>), grid, block, 0, s, Q, kv, O, st, g, kg, layer,
           scale, sp);
  else
    launch((attention_mfma_kernel<DH, NW, 2>), grid, block, 0, s, Q, kv, O, st, g, kg, layer,
           scale, sp);
}

// Merge of the key splits: O = sum_s f_s o_s / sum_s f_s l_s with
// f_s = exp(m_s - max m), splits taken in order.  One block of DH threads per
// (query row, head); the split loop is unrolled to its bound (16) so that all
// loads are in flight together.
template <int DH>
__global__ void __launch_bounds__(DH)
    attention_combine_kernel(bf16* __restrict__ O, KfStepGeom g, int H, AttnSplit sp) {
  constexpr int NSMAX = 16;
  const int h = blockIdx.x % H, rq = blockIdx.x / H, nqr = g.R - g.qoff;
  const int b = rq / nqr, i = g.qoff + (rq - b * nqr), e = threadIdx.x;
  const int row = b * g.R + i;
  const size_t base = (((size_t)b * H + h) * g.R + i) * sp.ns;
  float ms[NSMAX], ls[NSMAX], os[NSMAX];
#pragma unroll
  for (int s = 0; s < NSMAX; ++s) {
    const bool on = s < sp.ns;
    ms[s] = on ? sp.m[base + s] : -INFINITY;
    ls[s] = on ? sp.l[base + s] : 0.f;
    os[s] = on ? sp.o[(base + s) * DH + e] : 0.f;
  }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < NSMAX; ++s) M = fmaxf(M, ms[s]);
  float den = 0.f, acc = 0.f;
#pragma unroll
  for (int s = 0; s < NSMAX; ++s) {
    const float f = ms[s] == -INFINITY ? 0.f : __expf(ms[s] - M);
    den += f * ls[s];
    acc += f * os[s];
  }
  O[(size_t)row * H * DH + h * DH + e] = (bf16)(acc / den);
}

// ------------------------------------------------------- token selection
__device__ inline int out_index(const KfOutDesc& od, int C, int nr, int b, int j) {
  return od.gen_base >= 0 ? b * od.stride + (C + nr + j - od.gen_base) : b * od.stride + j;
}

// Greedy head decoding (Sec. 3.2, Appendix C.1): per noise row, the argmax
// over the vocabulary from the per-tile partials; exact ties to the lowest id.
__global__ void __launch_bounds__(256)
    argmax_select_kernel(const float* __restrict__ pval, const int* __restrict__ pidx, int n_tiles,
                         KfStepGeom g, const KfDevState* st, KfOutDesc od, int committed) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int rows = g.B * g.k;
  if (m >= rows) return;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  // The first 8 x 64 tiles (vocabularies up to 65536) are loaded together,
  // indices clamped into the row and masked below, so that the row costs one
  // memory round trip; wider rows finish in a loop.
  constexpr int U = 8;
  const float* prv = pval + (size_t)m * n_tiles;
  const int* pri = pidx + (size_t)m * n_tiles;
  float vv[U];
  int vi[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int t = lane + 64 * u, tc = t < n_tiles ? t : n_tiles - 1;
    vv[u] = prv[tc];
    vi[u] = pri[tc];
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const bool ok = lane + 64 * u < n_tiles;
    if (ok && (vv[u] > bv || (vv[u] == bv && vi[u] < bi))) { bv = vv[u]; bi = vi[u]; }
  }
  for (int t = lane + 64 * U; t < n_tiles; t += 64) {
    const float v = prv[t];
    const int i = pri[t];
    if (v > bv || (v == bv && i < bi)) { bv = v; bi = i; }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    float ov = __shfl_xor(bv, off, 64);
    int oi = __shfl_xor(bi, off, 64);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  if (lane == 0) {
    const int b = m / g.k, j = m % g.k;
    if (bi == 0x7fffffff) bi = 0;
    od.out[out_index(od, g.ctx(st, b) - committed, g.nr, b, j)] = bi;
    if (od.pend) od.pend[(size_t)g.slot(b) * od.pend_stride + j] = bi;
  }
}

// Inverse-CDF map (Appendix B, strict convention): smallest m with F_m > u,
// F the CDF of softmax(logits) in token-id order, evaluated as
// prefix(exp(l - max)) > u * Z in fp32 with a fixed chunked order.
// One workgroup of 1024 threads per sequence.
__global__ void __launch_bounds__(1024)
    icdf_select_kernel(const float* __restrict__ logits, int V, const float* __restrict__ u_in,
                       uint64_t seed, KfStepGeom g, const KfDevState* st, KfOutDesc od) {
  __shared__ float red[1024];
  __shared__ int found;
  const int b = blockIdx.x, t = threadIdx.x;
  const float* l = logits + (size_t)b * V;
  const int C = g.ctx(st, b);
  const float u = u_in ? u_in[b] : kf_noise_u(seed, g.slot(b), C + g.nr);
  const int chunk = (V + 1023) / 1024;
  const int lo = min(V, t * chunk), hi = min(V, lo + chunk);
  float mx = -INFINITY;
  for (int i = lo; i < hi; ++i) mx = fmaxf(mx, l[i]);
  red[t] = mx;
  __syncthreads();
  for (int s = 512; s > 0; s >>= 1) {
    if (t < s) red[t] = fmaxf(red[t], red[t + s]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float cs = 0.f;
  for (int i = lo; i < hi; ++i) cs += expf(l[i] - mx);
  red[t] = cs;
  if (t == 0) found = 0x7fffffff;
  __syncthreads();
  // inclusive scan of chunk sums (Hillis-Steele, fixed order)
  for (int s = 1; s < 1024; s <<= 1) {
    float add = (t >= s) ? red[t - s] : 0.f;
    __syncthreads();
    red[t] += add;
    __syncthreads();
  }
  const float Z = red[1023];
  const float target = u * Z;
  float run = (t > 0) ? red[t - 1] : 0.f;
  if (run <= target && red[t] > target) {
    // this chunk holds the crossing (at most one chunk satisfies both)
    int pick = hi - 1;
    for (int i = lo; i < hi; ++i) {
      run += expf(l[i] - mx);
      if (run > target) { pick = i; break; }
    }
    atomicMin(&found, pick);
  }
  __syncthreads();
  if (t == 0) {
    int tok = found;
    if (tok == 0x7fffffff) {  // rounding left F_V <= u: last token with q > 0
      tok = V - 1;
      for (int i = V - 1; i >= 0; --i)
        if (expf(l[i] - mx) > 0.f) { tok = i; break; }
    }
    od.out[out_index(od, C, g.nr, b, 0)] = tok;
    od.pend[(size_t)g.slot(b) * od.pend_stride] = tok;
  }
}

// Token rows of a whole-sequence forward laid out as N groups of k (the
// Future-1 rows of DoubleForward): row (b, t, j) takes token toks[b][t*k + j]
// at position t + shift + j into residual row b*n + off + t*k + j, with its
// LayerNorm partial sums, as embed_real_kernel does for a step's real rows.
template <typename T>
__global__ void __launch_bounds__(256)
    embed_group_kernel(float* __restrict__ X, T* __restrict__ Xh, float2* __restrict__ lnst,
                       const T* __restrict__ tok, const T* __restrict__ pos,
                       const int32_t* __restrict__ toks, int N, int k, int n, int off, int shift,
                       int d, int V, KfDevState* st) {
  const int r = blockIdx.x, nk = N * k;
  const int b = r / nk, q = r - b * nk, t = q / k, j = q - t * k;
  int tk = toks[(size_t)b * nk + q];
  if (tk < 0 || tk >= V) {
    if (threadIdx.x == 0) atomicOr(&st->err, 1);
    tk = 0;
  }
  const size_t row = (size_t)b * n + off + q;
  const T* te = tok + (size_t)tk * d;
  const T* pe = pos + (size_t)(t + shift + j) * d;
  const int grp = threadIdx.x;
  if (grp < d / 16) {
    float v[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) {
      const int e = grp * 16 + c;
      v[c] = to_f(te[e]) + to_f(pe[e]);
      X[row * d + e] = v[c];
      if constexpr (sizeof(T) == 2) Xh[row * d + e] = from_f<T>(v[c]);
    }
    lnst[row * (d / 16) + grp] = ln_group16_one(v);
  }
}

// ------------------------------------------------ teacher target selection
// Temperature-scaled inverse CDF over a whole vocabulary without the logits in
// HBM (Algorithm "Stage 1" teacher: targets = InverseCDF(softmax(l / tau), z)).
// The sampling head left, per row, the maximum M_t of x = l / tau in each
// 128-column tile and per 16-column group q the sum of exp(x - M_t).  With M
// the row maximum, the mass of tile t is w_t = exp(M_t - M) sum_q psub[t][q].
// One wavefront per row scans tile masses (lane L holds a contiguous run of
// tiles; an inclusive scan over the lanes keeps tile order), then the eight
// group masses of the crossing tile, then recomputes the crossing group's 16
// logits from the normalised hidden row and scans them: the result is the
// smallest column j with sum_{i <= j} p_i > u Z, the strict convention.  When
// rounding leaves no crossing (u Z at or above the total), every level takes
// its last element with positive mass, i.e. the last token with q > 0.
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// 8 consecutive elements of a compute-dtype row as floats
__device__ inline void load8f(const float* p, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ inline void load8f(const bf16* p, float (&x)[8]) {
  const uint4 v = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

template <typename T>
__global__ void __launch_bounds__(256)
    teacher_select_kernel(const float* __restrict__ pmax, const float* __restrict__ psub, int nT,
                          int V, const T* __restrict__ Xh, const float2* __restrict__ lnst,
                          const T* __restrict__ W, const float* __restrict__ c1,
                          const float* __restrict__ c2, int rms, int d, const float* __restrict__ tau,
                          const float* __restrict__ u, int row0, int M, int rows_per_seq,
                          int32_t* __restrict__ targets, KfDevState* st) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (m >= M) return;  // whole wavefront
  const int r = row0 + m;
  const float tb = tau[r / rows_per_seq];
  if (!(tb > 0.f && tb < INFINITY)) {
    if (lane == 0) {
      targets[r] = 0;
      atomicOr(&st->err, 2);
    }
    return;
  }
  const float it = 1.0f / tb;
  const float* pm = pmax + (size_t)m * nT;
  const float* ps = psub + (size_t)m * nT * 8;

  // level 1: tiles
  const int c = (nT + 63) / 64, t_lo = min(nT, lane * c), t_hi = min(nT, t_lo + c);
  float mx = -INFINITY;
  for (int t = t_lo; t < t_hi; ++t) mx = fmaxf(mx, pm[t]);
  mx = wave_max(mx);
  auto tile_w = [&](int t) {
    const float mt = pm[t];
    if (mt == -INFINITY) return 0.f;
    const float4 a = *reinterpret_cast<const float4*>(ps + (size_t)t * 8);
    const float4 b = *reinterpret_cast<const float4*>(ps + (size_t)t * 8 + 4);
    return __expf(mt - mx) * (((a.x + a.y) + (a.z + a.w)) + ((b.x + b.y) + (b.z + b.w)));
  };
  float ls = 0.f;
  for (int t = t_lo; t < t_hi; ++t) ls += tile_w(t);
  float incl = ls;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  const float Z = __shfl(incl, 63, 64);
  const float thr = u[r] * Z;
  const uint64_t cross = __ballot(incl > thr);
  const bool fall = cross == 0;
  int ls_lane;
  if (!fall) {
    ls_lane = __ffsll((unsigned long long)cross) - 1;
  } else {
    const uint64_t pos = __ballot(ls > 0.f);
    ls_lane = pos ? 63 - __clzll((unsigned long long)pos) : 0;
  }
  float run = __shfl(incl - ls, ls_lane, 64);  // mass before the lane's tiles
  int tstar = -1;
  {
    const int lo = min(nT, ls_lane * c), hi = min(nT, lo + c);
    float run_last = run;
    int t_last = lo;
    for (int t = lo; t < hi; ++t) {
      const float w = tile_w(t);
      if (!fall && run + w > thr) {
        tstar = t;
        break;
      }
      if (w > 0.f) {
        t_last = t;
        run_last = run;
      }
      run += w;
    }
    if (tstar < 0) {  // fallback, or rounding between the lane scan and the tile scan
      tstar = t_last;
      run = run_last;
    }
  }

  // level 2: the eight 16-column groups of tile tstar
  const float sc = __expf(pm[tstar] - mx);
  int qstar = -1;
  {
    float run_last = run;
    int q_last = 0;
    for (int q = 0; q < 8; ++q) {
      const float gq = sc * ps[(size_t)tstar * 8 + q];
      if (!fall && run + gq > thr) {
        qstar = q;
        break;
      }
      if (gq > 0.f) {
        q_last = q;
        run_last = run;
      }
      run += gq;
    }
    if (qstar < 0) {
      qstar = q_last;
      run = run_last;
    }
  }

  // level 3: recompute the group's 16 logits (four lanes per column) and scan
  const int j0 = tstar * kHeadTileN + qstar * 16;
  const int jj = lane >> 2, part = lane & 3, j = j0 + jj;
  float dot = 0.f;
  if (j < V) {
    const T* wr = W + (size_t)j * d;
    const T* xr = Xh + (size_t)r * d;
    for (int ch = part; ch < d / 8; ch += 4) {
      float a[8], b[8];
      load8f(wr + ch * 8, a);
      load8f(xr + ch * 8, b);
#pragma unroll
      for (int i = 0; i < 8; ++i) dot = fmaf(a[i], b[i], dot);
    }
  }
  dot += __shfl_xor(dot, 1, 64);
  dot += __shfl_xor(dot, 2, 64);
  // the row's LayerNorm statistics from its partial sums, as the head GEMM forms them
  float sa = 0.f;
  for (int i = lane; i < d / 16; i += 64) sa += lnst[(size_t)r * (d / 16) + i].x;
  sa = wave_sum(sa);
  const float mu = rms ? 0.f : sa / (float)d;
  float sb = 0.f;
  for (int i = lane; i < d / 16; i += 64) sb += ln_group_sq(lnst[(size_t)r * (d / 16) + i], mu);
  sb = wave_sum(sb);
  const float rstd = 1.0f / sqrtf(sb / (float)d + 1e-5f);
  float p = 0.f;
  if (j < V) {
    const float l = rstd * (dot - mu * c1[j]) + c2[j];
    p = __expf(l * it - pm[tstar]) * sc;
  }
  float pj = __shfl(p, 4 * (lane & 15), 64);  // lanes 0..15: column j0 + lane
  if (lane >= 16) pj = 0.f;
  float in16 = pj;
#pragma unroll
  for (int off = 1; off < 16; off <<= 1) {
    const float v = __shfl_up(in16, off, 64);
    if ((lane & 15) >= off) in16 += v;
  }
  const uint64_t hit = __ballot(lane < 16 && !fall && run + in16 > thr);
  int jstar;
  if (hit) {
    jstar = __ffsll((unsigned long long)hit) - 1;
  } else {
    const uint64_t pos = __ballot(lane < 16 && pj > 0.f);
    jstar = pos ? 63 - __clzll((unsigned long long)pos) : 0;
  }
  if (lane == 0) targets[r] = min(j0 + jstar, V - 1);
}

// End of step: the real rows' K/V become context (C += nr), for the batch or
// for each sequence slot of the step.
__global__ void commit_kernel(KfDevState* st, KfStepGeom g, int nr) {
  if (!g.map) {
    if (threadIdx.x == 0 && blockIdx.x == 0) st->C += nr;
    return;
  }
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < g.B) g.cs[g.map[b]] += nr;
}

__global__ void scatter_i32_kernel(int* dst, KfScatter u) {
  const int i = threadIdx.x;
  if (i < u.n) dst[u.idx[i]] = u.val[i];
}

// Admission of new sequences: their slots start from an empty context.
__global__ void seq_reset_kernel(KfStepGeom g) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < g.B) g.cs[g.map[b]] = 0;
}

__global__ void fill_noise_kernel(float* out, uint64_t seed, int B, int p0, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * n) return;
  out[i] = kf_noise_u(seed, i / n, p0 + i % n);
}

template <typename T>
__global__ void convert_kernel(const float* __restrict__ src, T* __restrict__ dst, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) dst[i] = from_f<T>(src[i]);
}

template <typename T>
__global__ void zero_kernel(T* dst, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) dst[i] = T(0);
}

__global__ void copy_f32_kernel(const float* __restrict__ src, float* __restrict__ dst, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) dst[i] = src[i];
}

inline unsigned grid_for(size_t n, unsigned block) {
  size_t gsz = (n + block - 1) / block;
  if (gsz > 65535u * 8u) gsz = 65535u * 8u;
  if (gsz == 0) gsz = 1;
  return (unsigned)gsz;
}

}  // namespace

// ------------------------------------------------------------ launchers
template <typename T>
hipError_t launch_embed_real(float* X, T* Xh, float2* lnst, const T* tok, const T* pos,
                             const int32_t* toks, int tok_stride, int toks_by_slot, KfStepGeom g,
                             int d, int V, KfDevState* st, hipStream_t s, const NoiseAhead* na) {
  const int blocks = g.B * g.nr + (na ? g.B * g.k : 0);
  if (blocks <= 0) return hipSuccess;
  const NoiseAhead none{nullptr, nullptr, nullptr, 0, 1, 0};
  launch(embed_real_kernel<T>, dim3(blocks), dim3(256), 0, s, X, Xh, lnst, tok, pos, toks,
                     tok_stride, toks_by_slot, g, d, V, st, na ? *na : none);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_noise_sinusoid_ahead(T* S, uint64_t seed, const double* omega, int B, int k,
                                       int N, int pass0, int npass, int d, hipStream_t s) {
  if (B <= 0 || k <= 0 || npass <= 0) return hipSuccess;
  launch(noise_sinusoid_ahead_kernel<T>, dim3(npass * B * k), dim3(256), 0, s, S, seed, omega, B,
         k, N, pass0, d);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_noise_sinusoid(T* S, const float* noise, uint64_t seed, const double* omega,
                                 KfStepGeom g, int d, const KfDevState* st, float* u_out,
                                 hipStream_t s) {
  if (g.k <= 0 || g.B <= 0) return hipSuccess;
  launch(noise_sinusoid_kernel<T>, dim3(g.B * g.k), dim3(256), 0, s, S, noise, seed,
                     omega, g, d, st, u_out);
  return hipGetLastError();
}

// Decode grids of 64 to 255 query blocks at d_head 64 (batch 6 to 21 at 12
// heads) run one workgroup of eight wavefronts per block instead of key
// splits of four-wavefront workgroups and their merge kernel: measured on the
// OWT-shaped model at batch 16, attention 43.2 -> 31.0 ms per generate (the
// generate 139.6 -> 130.5 ms).  Smaller grids keep the splits (batch 1 lost
// 4 % with eight wavefronts and no split), and grids of 256 blocks and more
// keep four wavefronts (batch 24 and 32 lost 5 %, batch 64 9 %, batch 256
// 15 % with eight).
constexpr int kWideMin = 64;

template <typename T>
hipError_t launch_attention(const T* Q, const T* kv, T* O, const KfDevState* st, KfStepGeom g,
                            KfKvGeom kg, int layer, const AttnSplit& ws, hipStream_t s) {
  if (g.B <= 0 || g.R - g.qoff <= 0) return hipSuccess;
  const float scale = 1.0f / sqrtf((float)kg.dh);
  if constexpr (sizeof(T) == 2) {
    // key splits: enough workgroups for ~512 in flight, each split at least
    // 128 keys of the full context, within the partial-state workspace
    const int base = g.B * kg.H * ((g.R - g.qoff + 15) / 16);
    int ns = 1;
    if (ws.o && base < 256) {
      ns = 512 / base;
      ns = ns < kg.T / 128 ? ns : kg.T / 128;
      ns = ns < 16 ? ns : 16;
      while (ns > 1 && (long long)g.B * kg.H * g.R * ns > ws.entries) --ns;
      if (ns < 1) ns = 1;
    }
    AttnSplit sp = ws;
    sp.ns = ns;
    dim3 grid(base * ns);
    switch (kg.dh) {
      case 32:
        launch_attention_mfma<32, 4>(grid, s, Q, kv, O, st, g, kg, layer, scale, sp);
        if (ns > 1)
          launch(attention_combine_kernel<32>, dim3(g.B * (g.R - g.qoff) * kg.H), dim3(32), 0, s,
                             O, g, kg.H, sp);
        break;
      case 64:
        if (ns > 1 && base >= kWideMin) {  // eight wavefronts, no key split
          sp.ns = 1;
          launch_attention_mfma<64, 8>(dim3(base), s, Q, kv, O, st, g, kg, layer, scale, sp);
          ns = 1;
          break;
        }
        if (ns == 1 && kg.T <= 128) {
          // contexts of at most 4 key tiles: two wavefronts, so that each
          // takes two tiles and its next-tile loads overlap its first tile
          // (LM1B-shaped batch 64: +0.6 %; one wavefront +0.1 %)
          launch_attention_mfma<64, 2>(grid, s, Q, kv, O, st, g, kg, layer, scale, sp);
          break;
        }
        launch_attention_mfma<64, 4>(grid, s, Q, kv, O, st, g, kg, layer, scale, sp);
        if (ns > 1)
          launch(attention_combine_kernel<64>, dim3(g.B * (g.R - g.qoff) * kg.H), dim3(64), 0, s,
                             O, g, kg.H, sp);
        break;
      case 128:
        launch_attention_mfma<128, 4>(grid, s, Q, kv, O, st, g, kg, layer, scale, sp);
        if (ns > 1)
          launch(attention_combine_kernel<128>, dim3(g.B * (g.R - g.qoff) * kg.H), dim3(128), 0, s,
                             O, g, kg.H, sp);
        break;
      default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  dim3 grid(g.B * kg.H, (g.R - g.qoff + 15) / 16);
  switch (kg.dh) {
    case 32:
      launch((attention_kernel<T, 32>), grid, dim3(256), 0, s, Q, kv, O, st, g, kg,
                         layer, scale);
      break;
    case 64:
      launch((attention_kernel<T, 64>), grid, dim3(256), 0, s, Q, kv, O, st, g, kg,
                         layer, scale);
      break;
    case 128:
      launch((attention_kernel<T, 128>), grid, dim3(256), 0, s, Q, kv, O, st, g, kg,
                         layer, scale);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_argmax_select(const float* pval, const int* pidx, int n_tiles, KfStepGeom g,
                                const KfDevState* st, KfOutDesc od, hipStream_t s, int committed) {
  int rows = g.B * g.k;
  if (rows <= 0) return hipSuccess;
  launch(argmax_select_kernel, dim3((rows + 3) / 4), dim3(256), 0, s, pval, pidx,
                     n_tiles, g, st, od, committed);
  return hipGetLastError();
}

hipError_t launch_icdf_select(const float* logits, int V, const float* u_in, uint64_t seed,
                              KfStepGeom g, const KfDevState* st, KfOutDesc od, hipStream_t s) {
  if (g.B <= 0) return hipSuccess;
  launch(icdf_select_kernel, dim3(g.B), dim3(1024), 0, s, logits, V, u_in, seed, g, st,
                     od);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_embed_group(float* X, T* Xh, float2* lnst, const T* tok, const T* pos,
                              const int32_t* toks, int B, int N, int k, int n, int off, int shift,
                              int d, int V, KfDevState* st, hipStream_t s) {
  if (B * N * k <= 0) return hipSuccess;
  launch(embed_group_kernel<T>, dim3(B * N * k), dim3(256), 0, s, X, Xh, lnst, tok, pos, toks, N,
         k, n, off, shift, d, V, st);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_teacher_select(const float* pmax, const float* psub, int n_tiles, int V,
                                 const T* Xh, const float2* lnst, const T* W, const float* c1,
                                 const float* c2, int rms, int d, const float* tau, const float* u,
                                 int row0, int M, int rows_per_seq, int32_t* targets, KfDevState* st,
                                 hipStream_t s) {
  if (M <= 0) return hipSuccess;
  launch(teacher_select_kernel<T>, dim3((M + 3) / 4), dim3(256), 0, s, pmax, psub, n_tiles, V, Xh,
         lnst, W, c1, c2, rms, d, tau, u, row0, M, rows_per_seq, targets, st);
  return hipGetLastError();
}

hipError_t launch_commit(KfDevState* st, KfStepGeom g, int nr, hipStream_t s) {
  launch(commit_kernel, dim3(g.map ? (g.B + 255) / 256 : 1), dim3(256), 0, s, st, g, nr);
  return hipGetLastError();
}

hipError_t launch_scatter_i32(int* dst, const KfScatter& u, hipStream_t s) {
  if (u.n <= 0) return hipSuccess;
  if (u.n > kScatterMax) return hipErrorInvalidValue;
  launch(scatter_i32_kernel, dim3(1), dim3(256), 0, s, dst, u);
  return hipGetLastError();
}

hipError_t launch_seq_reset(KfStepGeom g, hipStream_t s) {
  if (!g.map || g.B <= 0) return hipSuccess;
  launch(seq_reset_kernel, dim3((g.B + 255) / 256), dim3(256), 0, s, g);
  return hipGetLastError();
}

hipError_t launch_fill_noise(float* out, uint64_t seed, int B, int p0, int n, hipStream_t s) {
  if (B <= 0 || n <= 0) return hipSuccess;
  launch(fill_noise_kernel, dim3((B * n + 255) / 256), dim3(256), 0, s, out, seed, B,
                     p0, n);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_convert(const float* src, T* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  launch(convert_kernel<T>, dim3(grid_for(n, 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_zero(T* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  launch(zero_kernel<T>, dim3(grid_for(n, 256)), dim3(256), 0, s, dst, n);
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float* src, float* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  launch(copy_f32_kernel, dim3(grid_for(n, 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_zero_i32(int* dst, size_t n, hipStream_t s) { return launch_zero<int>(dst, n, s); }

#define KF_INST(T)                                                                                  \
  template hipError_t launch_embed_real<T>(float*, T*, float2*, const T*, const T*,               \
                                           const int32_t*, int, int, KfStepGeom, int, int,         \
                                           KfDevState*, hipStream_t, const NoiseAhead*);            \
  template hipError_t launch_noise_sinusoid_ahead<T>(T*, uint64_t, const double*, int, int, int,   \
                                                     int, int, int, hipStream_t);                  \
  template hipError_t launch_noise_sinusoid<T>(T*, const float*, uint64_t, const double*,          \
                                               KfStepGeom, int, const KfDevState*, float*,          \
                                               hipStream_t);                                        \
  template hipError_t launch_attention<T>(const T*, const T*, T*, const KfDevState*, KfStepGeom,   \
                                          KfKvGeom, int, const AttnSplit&, hipStream_t);            \
  template hipError_t launch_convert<T>(const float*, T*, size_t, hipStream_t);                    \
  template hipError_t launch_zero<T>(T*, size_t, hipStream_t);                                   \
  template hipError_t launch_embed_group<T>(float*, T*, float2*, const T*, const T*,              \
                                            const int32_t*, int, int, int, int, int, int, int, int, \
                                            KfDevState*, hipStream_t);                              \
  template hipError_t launch_teacher_select<T>(const float*, const float*, int, int, const T*,     \
                                               const float2*, const T*, const float*, const float*, \
                                               int, int, const float*, const float*, int, int, int, \
                                               int32_t*, KfDevState*, hipStream_t);
KF_INST(float)
KF_INST(bf16)
#undef KF_INST

}  // namespace kf
