// kf_blockattn.hip -- block-sparse attention of the training masks on gfx950.
//
// Appendix C.2 defines two masks over a sequence of N context tokens and k
// tokens per context position:
//   SingleForward M_S, queries and keys [context N | noise N*k]:
//     context row i sees context 0..i; noise token j of group t (t = 0..N-1)
//     sees context 0..t and tokens 0..j of its own group;
//   DoubleForward M_D, queries [Future-1 N*k | Future-2 N*k], keys
//     [context N | Future-1 N*k | Future-2 N*k]:
//     Future-1 token j of group t sees context 0..t and Future-1 tokens 0..j
//     of its group; Future-2 token j of group t sees context 0..t, all k
//     Future-1 tokens of its group and Future-2 tokens 0..j of its group.
// Every query row therefore sees at most three key intervals, one in each of
// the disjoint key regions (context, first noise block, second noise block).
// A workgroup owns 64 consecutive query rows (16 per wavefront) and walks only
// the union of their intervals, region by region, in 64-key tiles staged in
// LDS and shared by its four wavefronts.  A wavefront skips a tile that misses
// all of its rows and applies the per-element mask only on tiles that are not
// fully visible to all of them.  The work is O(|M|), not O((N + Nk)^2).
//
//   S^T = K Q^T on v_mfma_f32_16x16x32_bf16, keys as the A operand; a lane
//   ends up with query lq and keys 16g + 4gq + r (g, r = 0..3).
//   Online softmax in fp32 (base 2, the scale folded into the exponent).
//   O^T += V^T P^T: the lane's probabilities of key blocks 2c and 2c+1 are the
//   B operand of chunk c directly; the value tile is stored transposed in LDS
//   with its key slots permuted to the same order, so that each A operand is
//   one 16-byte LDS read.
#include <limits.h>
#include <math.h>

#include "../../include/kforcing.h"
#include "kf_internal.h"

namespace kf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kQB = 64;  // query rows per workgroup
constexpr int kKT = 64;  // keys per tile

// Visible key intervals [lo, hi) of one query row, one per key region
// (empty: lo >= hi).
struct Intervals {
  int lo[3], hi[3];
};

__device__ inline Intervals no_intervals() {
  Intervals v;
#pragma unroll
  for (int s = 0; s < 3; ++s) v.lo[s] = v.hi[s] = 0;
  return v;
}

__device__ inline Intervals row_intervals(int mask, int N, int k, int row) {
  Intervals v = no_intervals();
  if (mask == KF_MASK_SINGLE) {
    if (row < N) {
      v.hi[0] = row + 1;
    } else {
      const int q = row - N, t = q / k, j = q - t * k;
      v.hi[0] = t + 1;
      v.lo[1] = N + t * k;
      v.hi[1] = N + t * k + j + 1;
    }
  } else {
    const int nk1 = N * k;
    const bool f2 = row >= nk1;
    const int q = f2 ? row - nk1 : row, t = q / k, j = q - t * k;
    v.hi[0] = t + 1;
    v.lo[1] = N + t * k;
    v.hi[1] = f2 ? N + (t + 1) * k : N + t * k + j + 1;
    if (f2) {
      v.lo[2] = N + nk1 + t * k;
      v.hi[2] = N + nk1 + t * k + j + 1;
    }
  }
  return v;
}

// a[s] for a runtime s in 0..2 without indexing a register array
__device__ inline int pick(const int (&a)[3], int s) { return s == 0 ? a[0] : (s == 1 ? a[1] : a[2]); }

// LDS key slot of the 4-key group kg (keys 4kg..4kg+3 of a tile) in the
// transposed value tile: key 16g' + 4gq' + r of a 32-key chunk sits at slot
// 8gq' + 4g' + r, the order in which a lane holds its probabilities.
__device__ inline int v_slot(int kg) { return 32 * (kg >> 3) + 8 * (kg & 3) + 4 * ((kg >> 2) & 1); }

template <int DH>
struct TileRegs {
  static constexpr int NK = DH / 32;                  // 16-byte key chunks per thread
  static constexpr int NV = (4 * DH + 255) / 256;     // 4x4 value blocks per thread
  uint4 k[NK];
  uint2 v[NV][4];
};

// Global -> registers: keys t0..t0+63 of K and V ([key][DH] per head); keys at
// or past end read as zero.
template <int DH>
__device__ inline void load_tile(TileRegs<DH>& r, const bf16* Kh, const bf16* Vh, int t0, int end,
                                 int tid) {
#pragma unroll
  for (int i = 0; i < TileRegs<DH>::NK; ++i) {
    const int c = tid + 256 * i, key = t0 + c / (DH / 8), col = (c % (DH / 8)) * 8;
    r.k[i] = key < end ? *reinterpret_cast<const uint4*>(Kh + (size_t)key * DH + col)
                       : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < TileRegs<DH>::NV; ++i) {
    const int c = tid + 256 * i, kg = c & 15, cg = c >> 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int key = t0 + 4 * kg + e;
      r.v[i][e] = (c < 4 * DH && key < end)
                      ? *reinterpret_cast<const uint2*>(Vh + (size_t)key * DH + 4 * cg)
                      : make_uint2(0, 0);
    }
  }
}

// Registers -> LDS: keys as [key][DH + 8]; values transposed, [DH][64 + 8]
// with permuted key slots (v_slot).
template <int DH>
__device__ inline void store_tile(const TileRegs<DH>& r, bf16* sK, bf16* sV, int tid) {
  constexpr int KLD = DH + 8, VLD = kKT + 8;
#pragma unroll
  for (int i = 0; i < TileRegs<DH>::NK; ++i) {
    const int c = tid + 256 * i, key = c / (DH / 8), col = (c % (DH / 8)) * 8;
    *reinterpret_cast<uint4*>(sK + key * KLD + col) = r.k[i];
  }
#pragma unroll
  for (int i = 0; i < TileRegs<DH>::NV; ++i) {
    const int c = tid + 256 * i, kg = c & 15, cg = c >> 4;
    if (c < 4 * DH) {
      const uint2* x = r.v[i];
      bf16* dst = sV + (4 * cg) * VLD + v_slot(kg);
      // column e of the 4x4 block (keys 4kg..4kg+3, d_head 4cg..4cg+3)
      const uint2 c0 = make_uint2((x[0].x & 0xffffu) | (x[1].x << 16), (x[2].x & 0xffffu) | (x[3].x << 16));
      const uint2 c1 = make_uint2((x[0].x >> 16) | (x[1].x & 0xffff0000u), (x[2].x >> 16) | (x[3].x & 0xffff0000u));
      const uint2 c2 = make_uint2((x[0].y & 0xffffu) | (x[1].y << 16), (x[2].y & 0xffffu) | (x[3].y << 16));
      const uint2 c3 = make_uint2((x[0].y >> 16) | (x[1].y & 0xffff0000u), (x[2].y >> 16) | (x[3].y & 0xffff0000u));
      *reinterpret_cast<uint2*>(dst) = c0;
      *reinterpret_cast<uint2*>(dst + VLD) = c1;
      *reinterpret_cast<uint2*>(dst + 2 * VLD) = c2;
      *reinterpret_cast<uint2*>(dst + 3 * VLD) = c3;
    }
  }
}

template <int DH>
__global__ void __launch_bounds__(256)
    training_attention_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                              const bf16* __restrict__ V, bf16* __restrict__ O, int mask, int N,
                              int k, int nq, int nk, int BH, float scale_log2) {
  constexpr int NDC = DH / 32, NDB = DH / 16, KLD = DH + 8, VLD = kKT + 8;
  __shared__ __attribute__((aligned(16))) bf16 sK[2][kKT * KLD];
  __shared__ __attribute__((aligned(16))) bf16 sV[2][DH * VLD];

  // heaviest query blocks (latest rows) of every head first; consecutive
  // workgroups take consecutive heads
  const int nqb = (nq + kQB - 1) / kQB;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  const size_t bh = blockIdx.x % BH;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, gq = lane >> 4, lq = lane & 15;
  const int q0 = qb * kQB;
  const bf16* Kh = K + bh * (size_t)nk * DH;
  const bf16* Vh = V + bh * (size_t)nk * DH;

  // key ranges of the workgroup: per region, the union over its 64 rows
  int lo[3], hi[3], nt[3];
  {
    const Intervals v = q0 + lane < nq ? row_intervals(mask, N, k, q0 + lane) : no_intervals();
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      const bool ne = v.lo[s] < v.hi[s];
      int a = ne ? v.lo[s] : INT_MAX, b = ne ? v.hi[s] : 0;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        a = min(a, __shfl_xor(a, off, 64));
        b = max(b, __shfl_xor(b, off, 64));
      }
      lo[s] = a;
      hi[s] = b;
      nt[s] = b > a ? (b - a + kKT - 1) / kKT : 0;
    }
  }
  const int ntiles = nt[0] + nt[1] + nt[2];

  // this lane's query row; the wavefront's union (wlo, whi) and intersection
  // (ilo, ihi) of its 16 rows' intervals per region
  const int row = q0 + 16 * w + lq;
  const bool valid = row < nq;
  const Intervals iv = valid ? row_intervals(mask, N, k, row) : no_intervals();
  int wlo[3], whi[3], ilo[3], ihi[3];
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    const bool ne = iv.lo[s] < iv.hi[s];
    int a = ne ? iv.lo[s] : INT_MAX, b = ne ? iv.hi[s] : 0;
    int c = valid ? (ne ? iv.lo[s] : INT_MAX) : INT_MIN;
    int d = valid ? (ne ? iv.hi[s] : INT_MIN) : INT_MAX;
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
      a = min(a, __shfl_xor(a, off, 64));
      b = max(b, __shfl_xor(b, off, 64));
      c = max(c, __shfl_xor(c, off, 64));
      d = min(d, __shfl_xor(d, off, 64));
    }
    wlo[s] = a;
    whi[s] = b;
    ilo[s] = c;
    ihi[s] = d;
  }

  const bf16x8_t zero8 = {};
  bf16x8_t qf[NDC];
  {
    const bf16* qrow = Q + (bh * nq + (valid ? row : 0)) * DH + 8 * gq;
#pragma unroll
    for (int c = 0; c < NDC; ++c)
      qf[c] = valid ? __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * c))
                    : zero8;
  }

  // tile ti -> (region s, first key t0)
  auto tile = [&](int ti, int& s, int& t0) {
    s = ti < nt[0] ? 0 : (ti < nt[0] + nt[1] ? 1 : 2);
    const int first = s == 0 ? 0 : (s == 1 ? nt[0] : nt[0] + nt[1]);
    t0 = pick(lo, s) + (ti - first) * kKT;
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  TileRegs<DH> regs;
  {
    int s, t0;
    tile(0, s, t0);
    load_tile<DH>(regs, Kh, Vh, t0, pick(hi, s), tid);
    store_tile<DH>(regs, sK[0], sV[0], tid);
  }
  __syncthreads();

  for (int ti = 0; ti < ntiles; ++ti) {
    const int cur = ti & 1;
    int s, t0;
    tile(ti, s, t0);
    if (ti + 1 < ntiles) {
      int s1, t1;
      tile(ti + 1, s1, t1);
      load_tile<DH>(regs, Kh, Vh, t1, pick(hi, s1), tid);
    }
    if (t0 < pick(whi, s) && t0 + kKT > pick(wlo, s)) {
      const bf16* kb = sK[cur];
      const bf16* vb = sV[cur];
      f32x4_t sc[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        sc[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NDC; ++c) {
          const bf16x8_t a =
              *reinterpret_cast<const bf16x8_t*>(kb + (16 * g + lq) * KLD + 32 * c + 8 * gq);
          sc[g] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[c], sc[g], 0, 0, 0);
        }
      }
      // a tile serves its region's interval only (its last keys may spill
      // into the next region, which has tiles of its own)
      const bool full = t0 >= pick(ilo, s) && t0 + kKT <= pick(ihi, s);
      const int rlo = pick(iv.lo, s), rhi = pick(iv.hi, s);
      float x[16];
      float tmax = -INFINITY;
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = t0 + 16 * g + 4 * gq + r;
          float v = sc[g][r] * scale_log2;
          if (!full && (key < rlo || key >= rhi)) v = -INFINITY;
          x[4 * g + r] = v;
          tmax = fmaxf(tmax, v);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      const float m_new = fmaxf(m_run, tmax);
      const float ref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - ref);
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        x[i] = __builtin_amdgcn_exp2f(x[i] - ref);
        psum += x[i];
      }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db) o[db] *= alpha;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        bf16x8_t pf;
#pragma unroll
        for (int i = 0; i < 8; ++i) pf[i] = (bf16)x[8 * c + i];
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8_t a =
              *reinterpret_cast<const bf16x8_t*>(vb + (16 * db + lq) * VLD + 32 * c + 8 * gq);
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pf, o[db], 0, 0, 0);
        }
      }
    }
    if (ti + 1 < ntiles) store_tile<DH>(regs, sK[cur ^ 1], sV[cur ^ 1], tid);
    __syncthreads();
  }

  // lane: query lq, d_head 16db + 4gq + r
  float l = l_run;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (valid) {
    const float inv = 1.0f / l;
    bf16* orow = O + (bh * nq + row) * DH + 4 * gq;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const bf16 e0 = (bf16)(o[db][0] * inv), e1 = (bf16)(o[db][1] * inv);
      const bf16 e2 = (bf16)(o[db][2] * inv), e3 = (bf16)(o[db][3] * inv);
      const uint32_t w0 = (uint32_t)__builtin_bit_cast(uint16_t, e0) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, e1) << 16);
      const uint32_t w1 = (uint32_t)__builtin_bit_cast(uint16_t, e2) |
                          ((uint32_t)__builtin_bit_cast(uint16_t, e3) << 16);
      *reinterpret_cast<uint2*>(orow + 16 * db) = make_uint2(w0, w1);
    }
  }
}

}  // namespace

int training_attention_rows(int mask, int N, int k) {
  return mask == KF_MASK_SINGLE ? N + N * k : 2 * N * k;
}
int training_attention_keys(int mask, int N, int k) {
  return mask == KF_MASK_SINGLE ? N + N * k : N + 2 * N * k;
}

hipError_t launch_training_attention(int mask, int B, int H, int N, int k, int dh, const bf16* Q,
                                     const bf16* K, const bf16* V, bf16* O, float scale,
                                     hipStream_t s) {
  const int nq = training_attention_rows(mask, N, k);
  const int nk = training_attention_keys(mask, N, k);
  const int BH = B * H;
  const dim3 grid((unsigned)BH * ((nq + kQB - 1) / kQB));
  const float sl2 = scale * 1.4426950408889634f;
  switch (dh) {
    case 32:
      launch(training_attention_kernel<32>, grid, dim3(256), 0, s, Q, K, V, O, mask, N, k, nq, nk,
             BH, sl2);
      break;
    case 64:
      launch(training_attention_kernel<64>, grid, dim3(256), 0, s, Q, K, V, O, mask, N, k, nq, nk,
             BH, sl2);
      break;
    case 128:
      launch(training_attention_kernel<128>, grid, dim3(256), 0, s, Q, K, V, O, mask, N, k, nq,
             nk, BH, sl2);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace kf
