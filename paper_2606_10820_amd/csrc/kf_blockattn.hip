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
// the union of their intervals, region by region, in 64-key tiles that travel
// from HBM straight into an S-stage LDS ring (buffer loads with the lds
// modifier; keys past the interval read as zero) and are shared by its four
// wavefronts.  A wavefront skips a tile that misses all of its rows and
// applies the per-element mask only on tiles that are not fully visible to
// all of them.  The work is O(|M|), not O((N + Nk)^2).
//
//   S^T = K Q^T on v_mfma_f32_16x16x32_bf16, keys as the A operand; a lane
//   ends up with query lq and keys 16g + 4gq + r (g, r = 0..3).
//   Online softmax in fp32, base 2 with the scale folded into one FMA; the
//   running maximum is raised only when it grows by more than 2^8.
//   O^T += V^T P^T: the lane's probabilities of key blocks 2c and 2c+1 are the
//   B operand of chunk c directly, and the A operand comes from the natural
//   [key][d_head] value tile through transposing LDS reads (ds_read_b64_tr_b16)
//   whose row addresses put keys in that same order.
#include <limits.h>
#include <math.h>

#include <type_traits>
#include <utility>

#include "kforcing.h"
#include "kf_internal.h"
#include "kf_lds.h"

namespace kf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

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

// q / k for 0 <= q with q * k < 2^32, from km = ceil(2^32 / k) (km = 0 for
// k = 1): the rounded-up reciprocal errs by less than one in q / k there.
__device__ inline int div_k(int q, uint32_t km) {
  return km ? (int)__umulhi((uint32_t)q, km) : q;
}

__device__ inline Intervals row_intervals(int mask, int N, int k, uint32_t km, int row) {
  Intervals v = no_intervals();
  if (mask == KF_MASK_SINGLE) {
    if (row < N) {
      v.hi[0] = row + 1;
    } else {
      const int q = row - N, t = div_k(q, km), j = q - t * k;
      v.hi[0] = t + 1;
      v.lo[1] = N + t * k;
      v.hi[1] = N + t * k + j + 1;
    }
  } else {
    const int nk1 = N * k;
    const bool f2 = row >= nk1;
    const int q = f2 ? row - nk1 : row, t = div_k(q, km), j = q - t * k;
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

// Union [ulo, uhi) and intersection [ilo, ihi) per region of the intervals
// of query rows [a, b) (a < b <= rows).  Within each part of the query rows
// (single: context, noise; double: Future-1, Future-2) every endpoint is a
// non-decreasing function of the row and a region is either empty for all
// rows of the part or for none, so the first and last row of each part
// decide.  An empty union is [0, 0); an empty intersection has ilo > ihi.
__device__ inline void row_bounds(int mask, int N, int k, uint32_t km, int a, int b, int (&ulo)[3],
                                  int (&uhi)[3], int (&ilo)[3], int (&ihi)[3]) {
  const int split = mask == KF_MASK_SINGLE ? N : N * k;
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    ulo[s] = INT_MAX;
    uhi[s] = INT_MIN;
    ilo[s] = INT_MIN;
    ihi[s] = INT_MAX;
  }
  const int pa[2] = {a, max(a, split)}, pb[2] = {min(b, split), b};
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    if (pa[part] >= pb[part]) continue;
    const Intervals f = row_intervals(mask, N, k, km, pa[part]);
    const Intervals l = row_intervals(mask, N, k, km, pb[part] - 1);
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      if (f.lo[s] < f.hi[s]) {
        ulo[s] = min(ulo[s], f.lo[s]);
        uhi[s] = max(uhi[s], l.hi[s]);
        ilo[s] = max(ilo[s], l.lo[s]);
        ihi[s] = min(ihi[s], f.hi[s]);
      } else {
        ilo[s] = INT_MAX;
        ihi[s] = INT_MIN;
      }
    }
  }
#pragma unroll
  for (int s = 0; s < 3; ++s)
    if (ulo[s] >= uhi[s]) ulo[s] = uhi[s] = 0;
}

// a[s] for a runtime s in 0..2 without indexing a register array
__device__ inline int pick(const int (&a)[3], int s) { return s == 0 ? a[0] : (s == 1 ? a[1] : a[2]); }

template <int... I, typename F>
__device__ inline void static_for_impl(std::integer_sequence<int, I...>, F&& f) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F&& f) {
  static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

// Cross-lane reductions over the four 16-lane groups (lanes l, l^16, l^32, l^48)
// with the gfx950 permlane swaps (VALU, no LDS traffic).
// (scores are finite or -inf, so no NaN-quieting copies: plain v_max_f32)
__device__ inline float max2(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ inline float max_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
// max of three without the NaN-quieting copies that fmaxf adds (scores are
// finite or -inf here)
__device__ inline float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// Tile geometry.  A stage holds the K tile then the V tile, each [64 keys]
// [DH] bf16 in natural layout with 16-byte chunks permuted within each row:
// logical chunk c of key row r sits at chunk c ^ swz(r).  swz makes both
// readers conflict-free: the K reads (16 consecutive rows, one logical chunk)
// and the transposing V reads (8 consecutive rows, two adjacent chunks).
template <int DH, int S_>
struct Geo {
  static constexpr int ROWB = DH * 2;           // bytes per key row
  static constexpr int TILEB = kKT * ROWB;      // bytes of one K or V tile
  static constexpr int SEGW = TILEB / 1024 / 4; // 1 KB DMA segments per wavefront per tensor
  static constexpr int NCH = DH / 8;            // 16-byte chunks per row
  static constexpr int RP = 128 / DH;           // rows per 256 bytes (the 64 LDS banks)
  static constexpr int S = S_;                  // pipeline stages
  static constexpr int PER = 2 * SEGW;          // DMA instructions per wavefront per tile
  static constexpr int STAGEB = 2 * TILEB;
};

template <int DH>
__device__ inline int swz(int r) {
  constexpr int NCH = DH / 8, RP = 128 / DH;
  const int m = (r / RP) % NCH;
  return ((m & (NCH / 2 - 1)) << 1) | (m / (NCH / 2));
}

// Scalar geometry of one work item -- a head and a 64-row query block: the
// workgroup's key ranges as a tile sequence.  Tiles run over region 0, 1, 2,
// each from its union's first key in steps of 64; tile ti lies in region
// (ti >= b1) + (ti >= b2).
struct Item {
  int bh, q0, ntiles, b1, b2, lo0, dt1, dt2, hi0, de1, de2;
  __device__ int t0(int ti) const {
    return lo0 + kKT * ti + (ti >= b1 ? dt1 : 0) + (ti >= b2 ? dt2 : 0);
  }
  __device__ int end(int ti) const { return hi0 + (ti >= b1 ? de1 : 0) + (ti >= b2 ? de2 : 0); }
};

// Item t of the (head, query block) list: head t / nqb, its blocks heaviest
// (latest rows) first.
__device__ inline Item make_item(int t, int nqb, int mask, int N, int k, uint32_t km, int nq) {
  Item it;
  it.bh = t / nqb;
  it.q0 = (nqb - 1 - (t - it.bh * nqb)) * kQB;
  int lo[3], hi[3], ilo[3], ihi[3], nt[3];
  row_bounds(mask, N, k, km, it.q0, min(it.q0 + kQB, nq), lo, hi, ilo, ihi);
#pragma unroll
  for (int s = 0; s < 3; ++s) nt[s] = (hi[s] - lo[s] + kKT - 1) / kKT;
  it.ntiles = nt[0] + nt[1] + nt[2];
  it.b1 = nt[0];
  it.b2 = nt[0] + nt[1];
  it.lo0 = lo[0];
  it.dt1 = lo[1] - lo[0] - kKT * nt[0];
  it.dt2 = lo[2] - lo[1] - kKT * nt[1];
  it.hi0 = hi[0];
  it.de1 = hi[1] - hi[0];
  it.de2 = hi[2] - hi[1];
  return it;
}

template <int DH, int S>
__global__ void __launch_bounds__(256)
    training_attention_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                              const bf16* __restrict__ V, bf16* __restrict__ O, int mask, int N,
                              int k, uint32_t km, int nq, int ldk, int H, int BH, int o_inter,
                              float c2) {
  using G = Geo<DH, S>;
  constexpr int NDC = DH / 32, NDB = DH / 16;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[S * G::STAGEB];

  // Work order.  Workgroups are dealt to the 8 XCDs round-robin, so XCD x runs
  // workgroups x, x + 8, ...  Each XCD is given a contiguous run of the item
  // list (whole heads, one after another), so that the query blocks of one
  // head share its keys and values through that XCD's L2.
  const int nqb = (nq + kQB - 1) / kQB, total = BH * nqb;
  const int x8 = blockIdx.x & 7, j8 = blockIdx.x >> 3;
  const Item C = make_item(x8 * (total >> 3) + min(x8, total & 7) + j8, nqb, mask, N, k, km, nq);
  const int tid = threadIdx.x, lane = tid & 63, gq = lane >> 4, lq = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // DMA: segment w + 4i of a tile is LDS bytes [1024 (w + 4i), +1024); lane L
  // fills 16 of them, the chunk that the swizzle puts there
  uint32_t voff[G::SEGW];
#pragma unroll
  for (int i = 0; i < G::SEGW; ++i) {
    const int byte = (w + 4 * i) * 1024 + 16 * lane;
    const int r = byte / G::ROWB, pc = (byte % G::ROWB) / 16;
    voff[i] = r * G::ROWB + ((pc ^ swz<DH>(r)) * 16);
  }
  // LDS read offsets of this lane within a tile.  K (MFMA A of S^T): key row
  // 16g + lq, logical chunk 4c + gq.  V (transposing reads, MFMA A of O^T):
  // key row 32c + 4gq + lq/4 (+16 for the upper half of the k-slots), d_head
  // 16db + 4 (lq % 4), i.e. logical chunk 2db + (lq % 4) / 2, byte 8 (lq % 2).
  uint32_t kofs[NDC], vofs[NDB];
#pragma unroll
  for (int c = 0; c < NDC; ++c) kofs[c] = lq * G::ROWB + (((4 * c + gq) ^ swz<DH>(lq)) * 16);
  {
    const int r = 4 * gq + (lq >> 2);
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      vofs[db] = r * G::ROWB + (((2 * db + ((lq & 3) >> 1)) ^ swz<DH>(r)) * 16) + (lq & 1) * 8;
  }
  const bf16x8_t ones = {1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};

  // Tiles past the last one load nothing, so every wavefront issues the same
  // number of loads per tile.
  auto issue = [&](int ti, int stage) {
    const bool live = ti < C.ntiles;
    const int t0 = live ? C.t0(ti) : 0;
    const int rows = live ? min(C.end(ti) - t0, kKT) : 0;
    const size_t off = ((size_t)C.bh * ldk + t0) * DH;
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(K + off, rows * G::ROWB);
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(V + off, rows * G::ROWB);
    unsigned char* st = smem + stage * G::STAGEB;
#pragma unroll
    for (int i = 0; i < G::SEGW; ++i) dma16(rk, voff[i], 0, st + (w + 4 * i) * 1024);
#pragma unroll
    for (int i = 0; i < G::SEGW; ++i) dma16(rv, voff[i], 0, st + G::TILEB + (w + 4 * i) * 1024);
  };
#pragma unroll
  for (int j = 0; j < S - 1; ++j) issue(j, j);

  // this lane's query row, its Q fragment (MFMA B operand: d_head 32c + 8gq..+7)
  // and intervals; the wavefront's union (wlo, whi) and intersection (ilo, ihi)
  // of its 16 rows' intervals per region
  const int row = C.q0 + 16 * w + lq;
  const bool valid = row < nq;
  bf16x8_t qf[NDC];
  {
    const bf16* qrow = Q + ((size_t)C.bh * nq + (valid ? row : 0)) * DH + 8 * gq;
#pragma unroll
    for (int c = 0; c < NDC; ++c)
      qf[c] = valid ? __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(qrow + 32 * c))
                    : bf16x8_t{};
  }
  int wlo[3] = {0, 0, 0}, whi[3] = {0, 0, 0}, ilo[3] = {1, 1, 1}, ihi[3] = {0, 0, 0};
  if (C.q0 + 16 * w < nq)
    row_bounds(mask, N, k, km, C.q0 + 16 * w, min(C.q0 + 16 * w + 16, nq), wlo, whi, ilo, ihi);
  const Intervals iv = valid ? row_intervals(mask, N, k, km, row) : no_intervals();
  // running max m (log2 units); o = the unnormalised O^T; ls = the row sums of
  // P, formed by the MFMA against a block of ones (each element of ls is the
  // sum of this lane's query row over the bf16 probabilities that o uses)
  float m_run = -INFINITY;
  f32x4_t o[NDB], ls = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // per-region values of the current tile's region, updated where a region starts
  int cwlo = 0, cwhi = 0, cilo = 0, cihi = 0, rlo = 0, rhi = 0;
  for (int ti = 0; ti < C.ntiles; ++ti) {
    vm_wait<(S - 2) * G::PER>();  // this wavefront's part of tile ti has landed
    __builtin_amdgcn_s_barrier();  // ... and everyone's; stage (ti - 1) % S is free
    issue(ti + S - 1, (ti + S - 1) % S);
    if (ti == 0 || ti == C.b1 || ti == C.b2) {
      const int rs = (ti >= C.b1) + (ti >= C.b2);
      cwlo = pick(wlo, rs);
      cwhi = pick(whi, rs);
      cilo = pick(ilo, rs);
      cihi = pick(ihi, rs);
      rlo = pick(iv.lo, rs);
      rhi = pick(iv.hi, rs);
    }
    const int t0 = C.t0(ti);
    if (t0 < cwhi && t0 + kKT > cwlo) {  // some row of this wavefront sees the tile
      const uint32_t kb = lds_addr(smem + (ti % S) * G::STAGEB), vb = kb + G::TILEB;
      // S^T = K Q^T: lane holds query lq, keys 16g + 4gq + r
      u32x4 a[4][NDC];
      static_for<4>([&](auto gg) {
#pragma unroll
        for (int c = 0; c < NDC; ++c) a[gg][c] = ds_read16_off<gg * 16 * G::ROWB>(kb + kofs[c]);
      });
      lgkm_wait0();
      // value fragments of all 64 keys, in flight during the S MFMAs and the softmax
      u32x2 va[2][NDB], vc[2][NDB];
      static_for<2>([&](auto c) {
        static_for<NDB>([&](auto db) {
          va[c][db] = ds_read_tr16_off<c * 32 * G::ROWB>(vb + vofs[db]);
          vc[c][db] = ds_read_tr16_off<c * 32 * G::ROWB + 16 * G::ROWB>(vb + vofs[db]);
        });
      });
      f32x4_t sc[4];
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        sc[gg] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NDC; ++c) {
          pin(a[gg][c]);
          sc[gg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[gg][c]),
                                                           qf[c], sc[gg], 0, 0, 0);
        }
      }
      // mask: a tile serves its own region's interval only (its last keys may
      // spill into the next region, which has tiles of its own)
      if (!(t0 >= cilo && t0 + kKT <= cihi)) {
        const unsigned width = rhi > rlo ? (unsigned)(rhi - rlo) : 0u;
        const int base = t0 + 4 * gq - rlo;
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if ((unsigned)(base + 16 * gg + r) >= width) sc[gg][r] = -INFINITY;
      }
      float mx = max3(max3(sc[0][0], sc[0][1], sc[0][2]), max3(sc[0][3], sc[1][0], sc[1][1]),
                      max3(sc[1][2], sc[1][3], sc[2][0]));
      mx = max3(mx, max3(sc[2][1], sc[2][2], sc[2][3]), max3(sc[3][0], sc[3][1], sc[3][2]));
      mx = max3(mx, sc[3][3], sc[3][3]);
      mx = max_xor32(max_xor16(mx)) * c2;
      // rescale only when the row maximum grows by more than 2^8: probabilities
      // stay below 256, and the same reference serves numerator and denominator
      const bool grow = mx > m_run + 8.f;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float mn = grow ? mx : m_run;
        const float alpha = __builtin_amdgcn_exp2f(m_run - mn);
        ls *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) o[db] *= alpha;
        m_run = mn;
      }
      const float mref = m_run == -INFINITY ? 0.f : m_run;
      bf16x8_t pf[2];
#pragma unroll
      for (int gg = 0; gg < 4; ++gg)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          pf[gg >> 1][4 * (gg & 1) + r] =
              (bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(sc[gg][r], c2, -mref));
      ls = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[0], ls, 0, 0, 0);
      ls = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[1], ls, 0, 0, 0);
      // O^T += V^T P^T, keys 0..31 then 32..63
      lgkm_wait0();
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          pin(va[c][db]);
          pin(vc[c][db]);
          const u32x4 x = {va[c][db].x, va[c][db].y, vc[c][db].x, vc[c][db].y};
          o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, x), pf[c],
                                                          o[db], 0, 0, 0);
        }
    }
  }
  vm_wait<0>();  // loads issued for tiles past the last one

  // lane: query lq, d_head 16db + 4gq + r
  if (valid) {
    const float inv = __builtin_amdgcn_rcpf(ls[0]);  // ls >= 1: the row maximum's term
    // O: [B][H][nq][DH], or [B][nq][H][DH] (rows of a residual stream) with o_inter
    const int ob = C.bh / H, oh = C.bh - ob * H;
    bf16* orow = O + (o_inter ? (((size_t)ob * nq + row) * H + oh) * DH
                              : ((size_t)C.bh * nq + row) * DH) + 4 * gq;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const f32x2_t lo = {o[db][0] * inv, o[db][1] * inv}, hi = {o[db][2] * inv, o[db][3] * inv};
      *reinterpret_cast<uint2*>(orow + 16 * db) =
          make_uint2(__builtin_bit_cast(uint32_t, __builtin_convertvector(lo, bf16x2_t)),
                     __builtin_bit_cast(uint32_t, __builtin_convertvector(hi, bf16x2_t)));
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

namespace {

template <int DH, int S>
hipError_t launch_ta(int mask, int B, int H, int N, int k, const bf16* Q, const bf16* K,
                     const bf16* V, int ldk, bf16* O, int o_inter, float scale, hipStream_t s) {
  const int nq = training_attention_rows(mask, N, k);
  const int BH = B * H;
  const dim3 grid((unsigned)((long long)BH * ((nq + kQB - 1) / kQB)));  // one workgroup per item
  const float c2 = scale * 1.4426950408889634f;  // scale * log2(e)
  // q / k in the kernel by the rounded-up reciprocal: exact while q * k < 2^32
  if ((long long)nq * (k > 1 ? k : 1) >= (1LL << 32)) return hipErrorInvalidValue;
  const uint32_t km = k > 1 ? (uint32_t)(((1ULL << 32) + k - 1) / k) : 0u;
  launch(training_attention_kernel<DH, S>, grid, dim3(256), 0, s, Q, K, V, O, mask, N, k, km, nq,
         ldk, H, BH, o_inter, c2);
  return hipGetLastError();
}

hipError_t launch_ta_dh(int mask, int B, int H, int N, int k, int dh, const bf16* Q, const bf16* K,
                        const bf16* V, int ldk, bf16* O, int o_inter, float scale, hipStream_t s) {
  switch (dh) {
    case 32: return launch_ta<32, 3>(mask, B, H, N, k, Q, K, V, ldk, O, o_inter, scale, s);
    case 64: return launch_ta<64, 2>(mask, B, H, N, k, Q, K, V, ldk, O, o_inter, scale, s);
    case 128: return launch_ta<128, 2>(mask, B, H, N, k, Q, K, V, ldk, O, o_inter, scale, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_training_attention(int mask, int B, int H, int N, int k, int dh, const bf16* Q,
                                     const bf16* K, const bf16* V, bf16* O, float scale,
                                     hipStream_t s) {
  return launch_ta_dh(mask, B, H, N, k, dh, Q, K, V, training_attention_keys(mask, N, k), O, 0,
                      scale, s);
}

hipError_t launch_training_attention_seq(int mask, int B, int H, int N, int k, int dh, const bf16* Q,
                                         const bf16* K, const bf16* V, int ldk, bf16* O,
                                         float scale, hipStream_t s) {
  return launch_ta_dh(mask, B, H, N, k, dh, Q, K, V, ldk, O, 1, scale, s);
}

}  // namespace kf
