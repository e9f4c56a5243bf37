// kf_attn.h -- the bf16 block attention of one (sequence, head, block of 16
// query rows, key split) on MFMA, the body of the decode attention kernel.
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>

#include "kf_internal.h"

namespace kf {
namespace {

// Block attention on MFMA (bf16) for one (sequence, head, block of 16 query
// rows, key split) per workgroup; its NW wavefronts (four in the library: measured
// best from 64 keys up, and within 6 % of two waves at 16 keys; eight for
// mid-size decode grids, see kWideMin) take 32-key tiles of the split's key
// range round-robin and merge their online-softmax states through LDS at the
// end.
//   S^T = K Q^T   with v_mfma_f32_16x16x32_bf16: A = 16 keys x 32 d_head,
//                 B = 32 d_head x 16 queries.  MFMA row i of key group grp is
//                 key 8*(i/4) + 4*grp + i%4 of the tile, so the output rows a
//                 lane holds (4 per group, 2 groups) are 8 consecutive keys.
//   O^T += V^T P^T  A = 16 d_head x 32 keys read straight from the transposed
//                 value blocks (8 consecutive slots of a value row = two 8-byte
//                 loads), B = the lane's own 8 probabilities -- no data
//                 exchange between lanes.
// Each wavefront loads the K and V fragments of its next tile before working
// on the current one.  With ns > 1 key splits (grids too small to fill the
// chip), every split writes its unnormalised state (max m, sum l, o) for the
// combine kernel; the split count depends only on the shapes, not on the
// context length, so a captured step replays unchanged as C grows.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

__device__ inline bf16x8_t load8(const bf16* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(p));
}
// KV-cache reads are nontemporal: a decode pass streams every sequence's cache
// once, and keeping it from displacing other lines leaves the weights
// resident in the last-level cache from one pass to the next (measured 5 %
// faster per generate at both decode workloads).
__device__ inline bf16x8_t load8_stream(const bf16* p) {
  return __builtin_bit_cast(bf16x8_t, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p)));
}
__device__ inline u32x2_t load4_stream(const bf16* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
}

// The online softmax of one wavefront over the key tiles t0 = first, first +
// stride, ... < ke of (sequence b, head h) for the query rows q0 .. q0 + nq - 1
// of the step (nq <= 16): on return the lane (query lq = lane & 15, group
// gq = lane >> 4) holds the running maximum m_run and sum l_run of query lq
// (the same in its four groups) and o[db][r] = the unnormalised output of
// query lq at d_head index 16 db + 4 gq + r.
// Where a tile's KV page comes from: PT 0, no page table (sequence q owns
// pages q * np ...); PT 1, a page table of at most 64 pages per sequence, read
// once into one register per lane; PT 2, a longer page table, read per tile.
// The first two keep the tile loop free of dependent loads.
template <int DH, int PT>
__device__ __forceinline__ void attention_tiles(const bf16* __restrict__ Q, const bf16* __restrict__ kv,
                                                const KfDevState* st, const KfStepGeom& g,
                                                const KfKvGeom& kg, int layer, float scale, int b,
                                                int h, int q0, int nq, int first, int stride, int ke,
                                                float& m_run, float& l_run, f32x4_t (&o)[DH / 16]) {
  constexpr int KT = 32, NDC = DH / 32, NDB = DH / 16;
  const int d = kg.H * DH;
  const int lane = threadIdx.x & 63;
  const int gq = lane >> 4, lq = lane & 15;
  const int C = g.ctx(st, b), seq = g.slot(b);
  const int nkeys = C + q0 + nq;
  // Every load is unconditional, at an address clamped into the sequence's
  // pages, and the data past the end is masked where it is used: a select on
  // loaded data, or a load behind a branch, makes the compiler wait for the
  // loads in flight, and the next tile's loads would no longer overlap this
  // tile's arithmetic.  Query rows past nq load row nq - 1 (their outputs are
  // never stored).
  bf16x8_t qf[NDC];
  const bf16* qrow = Q + ((size_t)b * g.R + q0 + (lq < nq ? lq : nq - 1)) * d + h * DH + 8 * gq;
#pragma unroll
  for (int c = 0; c < NDC; ++c) qf[c] = load8(qrow + c * 32);
  const int qslot = C + q0 + lq;

  m_run = -INFINITY;
  l_run = 0.f;
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // The value fragment is kept as its two 8-byte halves and assembled in
  // tile(): an assembly at load time is a register copy that waits for the
  // load.
  struct Frag {
    bf16x8_t k[2][NDC];
    u32x2_t vlo[NDB], vhi[NDB];
  };
  // A tile starts at a multiple of 32 keys, so it lies in one KV page, and so
  // does the last key nkeys - 1 >= t0 that stands in for keys past the end
  // (their scores are masked to -inf).  Value slots past the end are read
  // from the same page and zeroed in tile() (their probability is 0, and
  // 0 * a stale NaN would not be).
  static_assert(kPage % KT == 0, "tiles do not straddle KV pages");
  const unsigned np = (unsigned)kg.T / kPage;
  unsigned pid = 0;
  if constexpr (PT == 1) pid = (unsigned)kg.ptab[(size_t)seq * np + ((unsigned)lane < np ? lane : np - 1)];
  auto page_of = [&](int t0) -> size_t {
    const unsigned j = (unsigned)t0 / kPage;
    unsigned pg;
    if constexpr (PT == 0) pg = (unsigned)seq * np + j;
    else if constexpr (PT == 1) pg = (unsigned)__builtin_amdgcn_readlane((int)pid, (int)j);
    else pg = (unsigned)kg.ptab[(size_t)seq * np + j];
    return (size_t)pg * kg.page_elems();
  };
  auto load = [&](int t0, Frag& f) {
    const bf16* page = kv + page_of(t0);
    const bf16* Kb = page + kg.head_off(layer, 0, h);
    const bf16* Vt = page + kg.head_off(layer, 1, h);
    const int pbase = t0 - t0 % kPage;
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      const int key = t0 + 8 * (lq >> 2) + 4 * grp + (lq & 3);
      const int kc = (key < nkeys ? key : nkeys - 1) - pbase;
#pragma unroll
      for (int c = 0; c < NDC; ++c) f.k[grp][c] = load8_stream(Kb + (size_t)kc * DH + c * 32 + 8 * gq);
    }
    const int kb = t0 + 8 * gq;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      // slots kb..kb+3 and kb+4..kb+7: two value blocks of this page
      f.vlo[db] = load4_stream(Vt + KfKvGeom::vt_off(kb - pbase, db * 16 + lq, DH));
      f.vhi[db] = load4_stream(Vt + KfKvGeom::vt_off(kb + 4 - pbase, db * 16 + lq, DH));
    }
  };
  auto tile = [&](int t0, const Frag& f) {
    bf16x8_t v[NDB];
#pragma unroll
    for (int db = 0; db < NDB; ++db)
      v[db] = __builtin_bit_cast(bf16x8_t, u32x4_t{f.vlo[db].x, f.vlo[db].y, f.vhi[db].x, f.vhi[db].y});
    if (t0 + KT > nkeys) {  // the ragged last tile: zero the value slots past the end
      const int kb = t0 + 8 * gq;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (kb + e >= nkeys) v[db][e] = (bf16)0.f;
    }
    f32x4_t s[2];
#pragma unroll
    for (int grp = 0; grp < 2; ++grp) {
      s[grp] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NDC; ++c)
        s[grp] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.k[grp][c], qf[c], s[grp], 0, 0, 0);
    }
    // this lane: query lq, keys t0 + 8*gq + 4*grp + r
    float p[8];
    float tmax = -INFINITY;
#pragma unroll
    for (int grp = 0; grp < 2; ++grp)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = t0 + 8 * gq + 4 * grp + r;
        const float v = (key <= qslot && key < nkeys) ? s[grp][r] * scale : -INFINITY;
        p[grp * 4 + r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float ref = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __expf(m_run - ref);
    float psum = 0.f;
    bf16x8_t pf;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = __expf(p[i] - ref);
      psum += p[i];
      pf[i] = (bf16)p[i];
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      o[db] *= alpha;
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v[db], pf, o[db], 0, 0, 0);
    }
  };

  // Ping-pong: the next tile loads while this one computes.  The last tile is
  // peeled off (no prefetch), so the loop body has no branch around a load.
  Frag fa, fb;
  int t0 = first;
  if (t0 >= ke) return;
  load(t0, fa);
  while (true) {
    if (t0 + stride >= ke) {
      tile(t0, fa);
      return;
    }
    load(t0 + stride, fb);
    tile(t0, fa);
    t0 += stride;
    if (t0 + stride >= ke) {
      tile(t0, fb);
      return;
    }
    load(t0 + stride, fa);
    tile(t0, fb);
    t0 += stride;
  }
}

template <int DH, int NW, int PT>
__device__ __forceinline__ void attention_block(const bf16* __restrict__ Q, const bf16* __restrict__ kv,
                                                bf16* __restrict__ O, const KfDevState* st,
                                                const KfStepGeom& g, const KfKvGeom& kg, int layer,
                                                float scale, const AttnSplit& sp, int b, int h,
                                                int qb, int split) {
  constexpr int QB = 16, KT = 32, NDB = DH / 16;
  const int H = kg.H, d = H * DH;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int gq = lane >> 4, lq = lane & 15;
  const int C = g.ctx(st, b);
  const int q0 = g.qoff + qb * QB, nq = min(QB, g.R - q0);
  const int nkeys = C + q0 + nq;
  const int chunk = ((nkeys + sp.ns - 1) / sp.ns + KT - 1) / KT * KT;
  const int ks = split * chunk, ke = min(nkeys, ks + chunk);
  float m_run, l_run;
  f32x4_t o[NDB];
  attention_tiles<DH, PT>(Q, kv, st, g, kg, layer, scale, b, h, q0, nq, ks + w * KT, NW * KT, ke,
                          m_run, l_run, o);

  // merge the wavefronts' partial states
  __shared__ float sm[NW][QB], sl[NW][QB];
  __shared__ float so[NW][QB][DH + 1];
  if (gq == 0) {
    sm[w][lq] = m_run;
    sl[w][lq] = l_run;
  }
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) so[w][lq][db * 16 + 4 * gq + r] = o[db][r];
  __syncthreads();
  constexpr int TPQ = 64 * NW / QB, EPT = DH / TPQ;  // threads per query row, elements each
  const int q = threadIdx.x / TPQ, e0 = (threadIdx.x % TPQ) * EPT;
  if (q < nq) {
    float M = -INFINITY;
#pragma unroll
    for (int i = 0; i < NW; ++i) M = fmaxf(M, sm[i][q]);
    float f[NW], den = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      f[i] = (sm[i][q] == -INFINITY) ? 0.f : __expf(sm[i][q] - M);
      den += f[i] * sl[i][q];
    }
    if (sp.ns == 1) {
      const float inv = 1.0f / den;
      bf16* orow = O + ((size_t)b * g.R + q0 + q) * d + h * DH + e0;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NW; ++i) acc += f[i] * so[i][q][e0 + e];
        orow[e] = (bf16)(acc * inv);
      }
    } else {
      const size_t ent = (((size_t)b * H + h) * g.R + q0 + q) * sp.ns + split;
      if (e0 == 0) {
        sp.m[ent] = M;
        sp.l[ent] = den;
      }
      float* orow = sp.o + ent * DH + e0;
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NW; ++i) acc += f[i] * so[i][q][e0 + e];
        orow[e] = acc;
      }
    }
  }
}


}  // namespace
}  // namespace kf
