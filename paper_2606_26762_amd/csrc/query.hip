// Query path of libprotokv for gfx950: pseudo-token synthesis and the
// mass-aware readout.
//
// Paper: Section "Residual Statistics and Pseudo-Token Interface" (pseudo
// tokens, mass-aware bias, Eq. attn_logit), Eq. pq and Appendix Algorithms
// "DecodeTopSResidualModes" and "ProtoKV Query-Time Pseudo-Token Decoding
// and Attention".
#include <mutex>
#include <type_traits>

#include "pkv_internal.h"

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t q_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float q_from_bf16(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// cos and sin of the rotary angle pos * inv (inv = theta^(-2i/D)): the angle
// in float64, whole turns taken off in float64, the rest (|r| <= pi) to
// float32 sincos.  Stream positions reach 10^6 and more, where a float32
// angle would already be off by tenths of a radian.
__device__ __forceinline__ void rope_cs(double pos, double inv, float& c, float& s) {
  const double a = pos * inv;
  const double turns = rint(a * 0.15915494309189535);  // 1 / (2 pi)
  const float r = (float)fma(-turns, 6.283185307179586, a);
  sincosf(r, &s, &c);
}

// Rotate-half rotation of the pair (x1 = dim i, x2 = dim i + D/2):
// lo = x1 c - x2 s, hi = x2 c + x1 s (float32, one rounding per operation).
__device__ __forceinline__ void rope_pair(float x1, float x2, float c, float s, float& lo, float& hi) {
  lo = x1 * c - x2 * s;
  hi = x2 * c + x1 * s;
}

// ---------------------------------------------------------------------------
// Exact top-S decoding of one PQ histogram.
//
// With eps = 1 the smoothed probability is (H[g][c]+1)/(n_res+C), so a code
// tuple's log-score sum_g log P(g, z_g) orders tuples exactly as the integer
// prod_g (H[g][z_g]+1); the denominator is common to every tuple.  Equal
// scores are ordered by the code tuple, lexicographically ascending.
//
// The beam of Alg. DecodeTopSResidualModes returns the exact top-S for any
// beam width B >= S (a prefix of a top-S tuple always ranks within the top S
// prefixes: otherwise S better prefixes, each completed with the same
// suffix, would give S better tuples).  So the beam here has width S: at
// subspace g the new beam is the best S of {prefix_i x rank_r}, taken by a
// merge over the prefixes (each prefix's extensions are already ordered by
// the codewords' rank (count desc, code asc)).
//
// Products are exact 192-bit integers (three 64-bit limbs): factors are
// < 2^24 and there are 8 of them.  Code tuples are packed one nibble per
// subspace, subspace 0 in the most significant nibble, so comparing packed
// values compares tuples lexicographically.
// ---------------------------------------------------------------------------
struct Big {
  uint64_t w0, w1, w2;  // little-endian limbs
};

__device__ __forceinline__ Big big_mul(const Big& a, uint32_t f) {
  Big r;
  unsigned __int128 t = (unsigned __int128)a.w0 * f;
  r.w0 = (uint64_t)t;
  t = (unsigned __int128)a.w1 * f + (uint64_t)(t >> 64);
  r.w1 = (uint64_t)t;
  t = (unsigned __int128)a.w2 * f + (uint64_t)(t >> 64);
  r.w2 = (uint64_t)t;
  return r;
}

// true if candidate (pa, ca) ranks before (pb, cb): larger product, then
// smaller packed code tuple.
__device__ __forceinline__ bool ranks_before(const Big& pa, uint32_t ca, const Big& pb, uint32_t cb) {
  if (pa.w2 != pb.w2) return pa.w2 > pb.w2;
  if (pa.w1 != pb.w1) return pa.w1 > pb.w1;
  if (pa.w0 != pb.w0) return pa.w0 > pb.w0;
  return ca < cb;
}

constexpr int SYN_P = 32;  // prototypes per workgroup (one wave: 32 x {keys, values})

// Per-thread beam state in dynamic LDS, planes [buf][entry][thread] so the
// 64 threads touch consecutive words: three 64-bit limbs and the packed code.
struct BeamView {
  uint64_t* w0;
  uint64_t* w1;
  uint64_t* w2;
  uint32_t* code;
  int S;
  __device__ __forceinline__ int at(int buf, int e, int tl) const { return (buf * S + e) * 64 + tl; }
};

__device__ void decode_top_s(const uint32_t* hist /* [G][CMAX] */, int C, int S, const BeamView& bv, int tl,
                             uint32_t* out_codes /* S */) {
  int nb = 1;
  int cur = 0;
  bv.w0[bv.at(0, 0, tl)] = 1;
  bv.w1[bv.at(0, 0, tl)] = 0;
  bv.w2[bv.at(0, 0, tl)] = 0;
  bv.code[bv.at(0, 0, tl)] = 0;
  for (int g = 0; g < G; ++g) {
    // rank the codewords of subspace g: count desc, code asc (top min(S, C))
    uint32_t h[CMAX];
#pragma unroll
    for (int c = 0; c < CMAX; ++c) h[c] = c < C ? hist[g * CMAX + c] : 0u;
    const int nr = S < C ? S : C;
    uint32_t rfac[SMAX], rcode[SMAX];
    uint32_t used = 0;
    for (int r = 0; r < nr; ++r) {
      int bc = -1;
      uint32_t bh = 0;
#pragma unroll
      for (int c = 0; c < CMAX; ++c) {
        const bool ok = c < C && !((used >> c) & 1u);
        if (ok && (bc < 0 || h[c] > bh)) { bc = c; bh = h[c]; }
      }
      used |= 1u << bc;
      rfac[r] = bh + 1u;
      rcode[r] = (uint32_t)bc;
    }
    // merge: row i = beam prefix i, column = rank
    int ptr[SMAX];
#pragma unroll
    for (int i = 0; i < SMAX; ++i) ptr[i] = 0;
    const int shift = 4 * (G - 1 - g);
    const int total = nb * nr;
    const int nout = S < total ? S : total;
    const int nxt = cur ^ 1;
    for (int o = 0; o < nout; ++o) {
      int bi = -1;
      Big bp{0, 0, 0};
      uint32_t bcode = 0;
      for (int i = 0; i < nb; ++i) {
        if (ptr[i] >= nr) continue;
        const int a = bv.at(cur, i, tl);
        Big p{bv.w0[a], bv.w1[a], bv.w2[a]};
        Big cand = big_mul(p, rfac[ptr[i]]);
        uint32_t code = bv.code[a] | (rcode[ptr[i]] << shift);
        if (bi < 0 || ranks_before(cand, code, bp, bcode)) { bi = i; bp = cand; bcode = code; }
      }
      ptr[bi] += 1;
      const int w = bv.at(nxt, o, tl);
      bv.w0[w] = bp.w0;
      bv.w1[w] = bp.w1;
      bv.w2[w] = bp.w2;
      bv.code[w] = bcode;
    }
    nb = nout;
    cur = nxt;
  }
  for (int s = 0; s < S; ++s) out_codes[s] = s < nb ? bv.code[bv.at(cur, s, tl)] : 0u;
}

// Register-resident exact top-S for prototypes whose residual count is at
// most 65534: every factor H+1 is below 2^16, so a product of 8 factors fits
// in 128 bits.  Same beam (width S) and merge order as decode_top_s.
struct U128 {
  uint64_t lo, hi;
};

__device__ __forceinline__ U128 mul_u128_u32(const U128& a, uint32_t f) {
  U128 r;
  const unsigned __int128 t0 = (unsigned __int128)a.lo * f;
  r.lo = (uint64_t)t0;
  r.hi = a.hi * (uint64_t)f + (uint64_t)(t0 >> 64);
  return r;
}

// Decoding, register path: LPB lanes (2 or 4) per (slot, K/V) beam,
// 64 / LPB beams per wave, for prototypes whose residual count is at most
// 65534 (every factor H+1 is below 2^16, so a product of the 8 factors fits
// in 128 bits) and S <= SM.  Lane q of a beam owns the prefixes e = q,
// q + LPB, ...  For each subspace the lanes rank the codewords (count desc,
// code asc) by counting, publish the top R = min(S, C) in order through LDS,
// and merge: S pops of the best row head (product desc, packed tuple asc),
// the best found in-lane and then with log2(LPB) DPP exchange steps across
// the beam's lanes; only the winning row advances.  Same beam (width S) and
// order as decode_top_s.
//
// With `centres` it also writes the float32 centre sum / n of the (slot,
// K/V) (IEEE division) and the slot's bias, for the readout's row forming.

// Exchanges within a quad of lanes (DPP quad_perm, no LDS round trip).
template <int CTRL>
__device__ __forceinline__ uint32_t qperm(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ uint64_t qperm64(uint64_t x) {
  return (uint64_t)qperm<CTRL>((uint32_t)x) | ((uint64_t)qperm<CTRL>((uint32_t)(x >> 32)) << 32);
}
constexpr int QP_XOR1 = 0xB1;  // lanes (1, 0, 3, 2)
constexpr int QP_XOR2 = 0x4E;  // lanes (2, 3, 0, 1)
// value of lane SRC of this lane's quad
template <int LPB, int SRC>
__device__ __forceinline__ uint32_t group_bcast(uint32_t x) {
  static_assert(LPB == 4, "quad broadcast");
  return qperm<SRC * 0x55>(x);
}

// (pa, ca) ranks before (pb, cb), without branches
__device__ __forceinline__ bool before128b(const U128& pa, uint32_t ca, const U128& pb, uint32_t cb) {
  const bool gh = pa.hi > pb.hi, eh = pa.hi == pb.hi, gl = pa.lo > pb.lo, el = pa.lo == pb.lo;
  return gh | (eh & (gl | (el & (ca < cb))));
}
__device__ __forceinline__ uint64_t sel64(bool t, uint64_t a, uint64_t b) {
  const uint64_t m = 0ull - (uint64_t)t;
  return (a & m) | (b & ~m);
}
__device__ __forceinline__ uint32_t sel32(bool t, uint32_t a, uint32_t b) {
  const uint32_t m = 0u - (uint32_t)t;
  return (a & m) | (b & ~m);
}

// Product helpers of the decode merge: 64-bit or 128-bit unsigned products.
template <typename P> __device__ __forceinline__ P pt_from(uint32_t x);
template <> __device__ __forceinline__ uint64_t pt_from<uint64_t>(uint32_t x) { return x; }
template <> __device__ __forceinline__ U128 pt_from<U128>(uint32_t x) { return U128{x, 0ull}; }
__device__ __forceinline__ uint64_t pt_mul(uint64_t a, uint32_t f) { return a * f; }
__device__ __forceinline__ U128 pt_mul(const U128& a, uint32_t f) { return mul_u128_u32(a, f); }
__device__ __forceinline__ bool pt_before(uint64_t pa, uint32_t ca, uint64_t pb, uint32_t cb) {
  return (pa > pb) | ((pa == pb) & (ca < cb));
}
__device__ __forceinline__ bool pt_before(const U128& pa, uint32_t ca, const U128& pb, uint32_t cb) {
  return before128b(pa, ca, pb, cb);
}
__device__ __forceinline__ uint64_t pt_sel(bool t, uint64_t a, uint64_t b) { return sel64(t, a, b); }
__device__ __forceinline__ U128 pt_sel(bool t, const U128& a, const U128& b) {
  return U128{sel64(t, a.lo, b.lo), sel64(t, a.hi, b.hi)};
}
template <int CTRL> __device__ __forceinline__ uint64_t pt_perm(uint64_t x) { return qperm64<CTRL>(x); }
template <int CTRL> __device__ __forceinline__ U128 pt_perm(const U128& x) {
  return U128{qperm64<CTRL>(x.lo), qperm64<CTRL>(x.hi)};
}

// The beam merge of k_decode4 for one product type P (uint64_t when every
// product of the wave's beams fits in 64 bits, else U128): products of the
// factors H+1 compare exactly either way.
template <int SM, int LPB, typename P>
__device__ __forceinline__ void decode_beam(uint32_t (*s_rank)[CMAX], const uint32_t* hist, bool mine, int S,
                                            int C, int q, int bq, uint32_t* out) {
  constexpr int E = SM / LPB;        // prefixes per lane
  constexpr int KPL = CMAX / LPB;    // codewords per lane
  const int R = S < C ? S : C;
  P pp[E];
  uint32_t pc[E];
#pragma unroll
  for (int j = 0; j < E; ++j) {
    pp[j] = pt_from<P>((q == 0 && j == 0) ? 1u : 0u);
    pc[j] = 0;
  }
  int nb = 1;
  // this lane's counts of subspace g, loaded one subspace ahead
  uint4 hnext[KPL / 4];
#pragma unroll
  for (int v4 = 0; v4 < KPL / 4; ++v4)
    hnext[v4] = mine ? reinterpret_cast<const uint4*>(hist)[q * (KPL / 4) + v4] : make_uint4(0, 0, 0, 0);
  for (int g = 0; g < G; ++g) {
    uint4 hcur[KPL / 4];
#pragma unroll
    for (int v4 = 0; v4 < KPL / 4; ++v4) {
      hcur[v4] = hnext[v4];
      hnext[v4] = mine && g + 1 < G ? reinterpret_cast<const uint4*>(hist + (g + 1) * CMAX)[q * (KPL / 4) + v4]
                                    : make_uint4(0, 0, 0, 0);
    }
    // keys of codewords KPL q .. KPL q + KPL - 1: (count << 4 | (15 - c)) + 1,
    // larger = better, 0 = absent
    uint32_t key[KPL];
#pragma unroll
    for (int v4 = 0; v4 < KPL / 4; ++v4) {
      const uint4 h4 = hcur[v4];
      const uint32_t hv[4] = {h4.x, h4.y, h4.z, h4.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = KPL * q + 4 * v4 + i;
        key[4 * v4 + i] = c < C ? ((hv[i] << 4) | (uint32_t)(15 - c)) + 1u : 0u;
      }
    }
    // ranks of the 16 keys (unique: the code is in the low bits)
    if constexpr (LPB == 2) {
      // each lane sorts its 8 keys descending (bitonic network), then one
      // bitonic half-cleaner across the pair (lane 0 keeps the larger of
      // key[k] and the partner's key[7 - k], lane 1 the smaller) and a
      // bitonic merge of 8 leave lane 0 with ranks 0..7 and lane 1 with
      // ranks 8..15, both in order
      auto cx = [&](int a, int b, bool desc) {
        const uint32_t x = key[a], y = key[b];
        const uint32_t hi = x > y ? x : y, lo = x > y ? y : x;
        key[a] = desc ? hi : lo;
        key[b] = desc ? lo : hi;
      };
#pragma unroll
      for (int k = 2; k <= KPL; k <<= 1)
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
          for (int i = 0; i < KPL; ++i)
            if ((i ^ j) > i) cx(i, i ^ j, (i & k) == 0);
      uint32_t t[KPL];
#pragma unroll
      for (int k = 0; k < KPL; ++k) t[k] = qperm<QP_XOR1>(key[KPL - 1 - k]);
#pragma unroll
      for (int k = 0; k < KPL; ++k) {
        const uint32_t hi = key[k] > t[k] ? key[k] : t[k], lo = key[k] > t[k] ? t[k] : key[k];
        key[k] = q == 0 ? hi : lo;
      }
#pragma unroll
      for (int j = KPL >> 1; j > 0; j >>= 1)
#pragma unroll
        for (int i = 0; i < KPL; ++i)
          if ((i ^ j) > i) cx(i, i ^ j, true);
#pragma unroll
      for (int i = 0; i < KPL; ++i)
        if (key[i] != 0u && q * KPL + i < R) s_rank[bq][q * KPL + i] = key[i];
    } else {
      int rk[KPL];
#pragma unroll
      for (int i = 0; i < KPL; ++i) rk[i] = 0;
#pragma unroll
      for (int i2 = 0; i2 < KPL; ++i2) {
        const uint32_t others[4] = {group_bcast<LPB, 0>(key[i2]), group_bcast<LPB, 1>(key[i2]),
                                    group_bcast<LPB, 2>(key[i2]), group_bcast<LPB, 3>(key[i2])};
#pragma unroll
        for (int src = 0; src < LPB; ++src)
#pragma unroll
          for (int i = 0; i < KPL; ++i) rk[i] += others[src] > key[i] ? 1 : 0;
      }
#pragma unroll
      for (int i = 0; i < KPL; ++i)
        if (key[i] != 0u && rk[i] < R) s_rank[bq][rk[i]] = key[i];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int shift = 4 * (G - 1 - g);
    if (g == 0) {
      // one prefix (the empty tuple): the beam is the ranks themselves
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const int e = q + LPB * j;
        const uint32_t ke = s_rank[bq][e < R ? e : 0];
        pp[j] = pt_from<P>(e < R ? ((ke - 1u) >> 4) + 1u : 0u);
        pc[j] = e < R ? (15u - ((ke - 1u) & 15u)) << shift : 0u;
      }
      nb = S < R ? S : R;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      continue;
    }
    const uint32_t k0 = s_rank[bq][0];
    // row heads: prefix e = q + LPB j times rank ptr[j]
    int ptr[E];
    P hp[E];
    uint32_t hc[E];
#pragma unroll
    for (int j = 0; j < E; ++j) {
      ptr[j] = 0;
      const bool ok = q + LPB * j < nb;
      hp[j] = ok ? pt_mul(pp[j], ((k0 - 1u) >> 4) + 1u) : pt_from<P>(0u);
      hc[j] = ok ? (pc[j] | ((15u - ((k0 - 1u) & 15u)) << shift)) : 0xFFFFFFFFu;
    }
    const int nout = S < nb * R ? S : nb * R;
    P np[E];
    uint32_t nc[E];
#pragma unroll
    for (int j = 0; j < E; ++j) { np[j] = pt_from<P>(0u); nc[j] = 0; }
#pragma unroll
    for (int o = 0; o < SM; ++o) {
      if (o < nout) {
        // best head of this lane (product 0 = exhausted row)
        P bv = hp[0];
        uint32_t bc = hc[0];
        int bj = 0;
#pragma unroll
        for (int j = 1; j < E; ++j) {
          const bool t = pt_before(hp[j], hc[j], bv, bc);
          bv = pt_sel(t, hp[j], bv);
          bc = sel32(t, hc[j], bc);
          bj = t ? j : bj;
        }
        uint32_t who = (uint32_t)(q * E + bj);
        // best of the beam's lanes
#pragma unroll
        for (int x = 0; x < (LPB == 4 ? 2 : 1); ++x) {
          P ov;
          uint32_t oc, ow;
          if (x == 0) {
            ov = pt_perm<QP_XOR1>(bv);
            oc = qperm<QP_XOR1>(bc); ow = qperm<QP_XOR1>(who);
          } else {
            ov = pt_perm<QP_XOR2>(bv);
            oc = qperm<QP_XOR2>(bc); ow = qperm<QP_XOR2>(who);
          }
          const bool t = pt_before(ov, oc, bv, bc);
          bv = pt_sel(t, ov, bv);
          bc = sel32(t, oc, bc);
          who = sel32(t, ow, who);
        }
        {
          const bool rec = (o % LPB) == q;
          np[o / LPB] = pt_sel(rec, bv, np[o / LPB]);
          nc[o / LPB] = sel32(rec, bc, nc[o / LPB]);
        }
        // the winning row moves to its next rank: one product, then selects
        const bool iwin = (int)(who / E) == q;
        const int j = (int)(who % E);
        int pj = ptr[0];
        P base = pp[0];
        uint32_t bcode = pc[0];
#pragma unroll
        for (int jj = 1; jj < E; ++jj) {
          const bool t = jj == j;
          pj = t ? ptr[jj] : pj;
          base = pt_sel(t, pp[jj], base);
          bcode = sel32(t, pc[jj], bcode);
        }
        pj += 1;
        const bool more = pj < R;
        const uint32_t kk = s_rank[bq][more ? pj : 0];
        const P nh = pt_sel(more, pt_mul(base, ((kk - 1u) >> 4) + 1u), pt_from<P>(0u));
        const uint32_t ncode = more ? (bcode | ((15u - ((kk - 1u) & 15u)) << shift)) : 0xFFFFFFFFu;
#pragma unroll
        for (int jj = 0; jj < E; ++jj) {
          const bool t = iwin && jj == j;
          ptr[jj] = t ? pj : ptr[jj];
          hp[jj] = pt_sel(t, nh, hp[jj]);
          hc[jj] = sel32(t, ncode, hc[jj]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < E; ++j) { pp[j] = np[j]; pc[j] = nc[j]; }
    nb = nout;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  if (mine) {
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int o = q + LPB * j;
      if (o < S) out[o] = o < nb ? pc[j] : 0u;
    }
    if (q == 0) out[SMAX] = 0u;
  }
}

template <int SM, int LPB>
__global__ __launch_bounds__(256) void k_decode4(Dims dm, Workspace ws, int sid, int n_active, int centres) {
  static_assert(LPB == 2 || LPB == 4, "lanes per beam");
  constexpr int E = SM / LPB;        // prefixes per lane
  constexpr int BPW = 64 / LPB;      // beams per wave
  constexpr int KPL = CMAX / LPB;    // codewords per lane
  __shared__ uint32_t s_rank[4][BPW][CMAX];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane & (LPB - 1), bq = lane / LPB;
  const int beam = (blockIdx.x * 4 + wave) * BPW + bq;  // ((unit * n_active + slot) * 2 + K/V)
  const bool bvalid = beam < dm.units * n_active * 2;
  const int kv = beam & 1, up = bvalid ? beam >> 1 : 0;
  const int u = up / n_active, p = up % n_active;
  const size_t unit = (size_t)sid * dm.units + u;
  const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  uint32_t* out = ws.pcodes + (((size_t)u * dm.K + p) * 2 + kv) * PCW;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0;
  const int S = dm.S, C = dm.C;
  const bool nores = !pq || m.n_res == 0;
  if (bvalid && q == 0 && nores) out[SMAX] = 1u;
  if (bvalid && centres && q == 0) {
    if (kv == 0) {
      const bool mb = (dm.flags & PROTOKV_FLAG_MASS_BIAS) != 0;
      ws.pbias[(size_t)u * dm.K + p] = mb ? logf((float)m.n) : 0.f;
      // tau_k in the key record's spare word: the readout rotates the
      // slot's formed pseudo-keys at it
      out[SMAX + 1] = (uint32_t)m.tau;
    } else {
      // n in the value record's spare word: the readout divides the slot's
      // sums by it
      out[SMAX + 1] = m.n;
    }
  }
  // this path decodes the beam (uniform within the beam's lanes)
  const bool mine = bvalid && !nores && m.n_res <= 65534u && S <= SM;
  const uint32_t* hist = reinterpret_cast<const uint32_t*>(row + (kv ? ROW_HV : ROW_HK));
  // every product the merge forms is at most prod_g max_c (H[g][c] + 1) (the
  // beam's top tuple); when that fits in 64 bits for all of the wave's
  // beams the merge runs on 64-bit products
  bool fits = true;
  if (mine) {
    uint64_t bound = 1;
    bool ovf = false;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint32_t mx = 0;
#pragma unroll
      for (int v4 = 0; v4 < KPL / 4; ++v4) {
        const uint4 h4 = reinterpret_cast<const uint4*>(hist + g * CMAX)[q * (KPL / 4) + v4];
        mx = max(mx, max(max(h4.x, h4.y), max(h4.z, h4.w)));
      }
      mx = max(mx, qperm<QP_XOR1>(mx));
      if (LPB == 4) mx = max(mx, qperm<QP_XOR2>(mx));
      ovf |= __builtin_mul_overflow(bound, (uint64_t)mx + 1u, &bound);
    }
    fits = !ovf;
  }
  if (__all(fits))
    decode_beam<SM, LPB, uint64_t>(s_rank[wave], hist, mine, S, C, q, bq, out);
  else
    decode_beam<SM, LPB, U128>(s_rank[wave], hist, mine, S, C, q, bq, out);
}

// Decoding, one lane per (slot, K/V) beam (S <= 8): the same beam search
// as decode_beam, with each subspace's merge done by sorting networks in
// registers.  For S <= 8, the top S of the (prefix i, rank j) products can
// only come from pairs with (i + 1)(j + 1) <= 8 (every pair (i', j') with
// i' <= i, j' <= j ranks at least as high: both lists are sorted, and equal
// products fall back to the packed tuple, whose prefix nibbles lead): the
// column j = 0 (8 prefixes), j = 1 (4), j = 2 and 3 (2 each), and prefix 0
// with ranks 4..7.  These sorted lists are merged into the running top 8 by
// a half-cleaner and a bitonic merger each.

// (pa, ca) and (pb, cb) in rank order (product desc, packed tuple asc)
template <typename P>
__device__ __forceinline__ void cx_rank(P& pa, uint32_t& ca, P& pb, uint32_t& cb) {
  const bool sw = pt_before(pb, cb, pa, ca);
  const P tp = pa;
  const uint32_t tc = ca;
  pa = pt_sel(sw, pb, pa);
  ca = sel32(sw, cb, ca);
  pb = pt_sel(sw, tp, pb);
  cb = sel32(sw, tc, cb);
}
// (pa, ca) becomes the first in rank order of a and b
template <typename P>
__device__ __forceinline__ void keep_first(P& pa, uint32_t& ca, const P& pb, uint32_t cb) {
  const bool sw = pt_before(pb, cb, pa, ca);
  pa = pt_sel(sw, pb, pa);
  ca = sel32(sw, cb, ca);
}
// bitonic sequence of 8 -> rank order
template <typename P>
__device__ __forceinline__ void bmerge8(P (&p)[8], uint32_t (&c)[8]) {
#pragma unroll
  for (int j = 4; j > 0; j >>= 1)
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if ((i & j) == 0) cx_rank(p[i], c[i], p[i + j], c[i + j]);
}
// (p, c) <- the first 8 in rank order of (p, c) and (lp, lc), both sorted
template <int K, typename P>
__device__ __forceinline__ void merge_top8(P (&p)[8], uint32_t (&c)[8], const P (&lp)[K], const uint32_t (&lc)[K]) {
#pragma unroll
  for (int i = 8 - K; i < 8; ++i) keep_first(p[i], c[i], lp[7 - i], lc[7 - i]);
  bmerge8(p, c);
}
// 32-bit keys (unique, larger first): a[0..7] sorted descending
__device__ __forceinline__ void sort8_desc(uint32_t* a) {
#pragma unroll
  for (int k = 2; k <= 8; k <<= 1)
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if ((i ^ j) > i) {
          const uint32_t x = a[i], y = a[i ^ j];
          const uint32_t hi = x > y ? x : y, lo = x > y ? y : x;
          const bool desc = (i & k) == 0;
          a[i] = desc ? hi : lo;
          a[i ^ j] = desc ? lo : hi;
        }
}

template <typename P>
__device__ __forceinline__ void decode_beam1(const uint32_t* hist, bool mine, int S, int C, uint32_t* out) {
  const int R = S < C ? S : C;
  P pp[8];
  uint32_t pc[8];
  int nb = 0;
  uint4 hnext[4];
#pragma unroll
  for (int v4 = 0; v4 < 4; ++v4) hnext[v4] = mine ? reinterpret_cast<const uint4*>(hist)[v4] : make_uint4(0, 0, 0, 0);
  for (int g = 0; g < G; ++g) {
    uint4 hcur[4];
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      hcur[v4] = hnext[v4];
      hnext[v4] = mine && g + 1 < G ? reinterpret_cast<const uint4*>(hist + (g + 1) * CMAX)[v4] : make_uint4(0, 0, 0, 0);
    }
    // keys (count << 4 | (15 - c)) + 1, larger = better, 0 = absent; the
    // first 8 in order: both halves sorted, then a half-cleaner and a merger
    uint32_t key[16];
#pragma unroll
    for (int v4 = 0; v4 < 4; ++v4) {
      const uint32_t hv[4] = {hcur[v4].x, hcur[v4].y, hcur[v4].z, hcur[v4].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = 4 * v4 + i;
        key[c] = c < C ? ((hv[i] << 4) | (uint32_t)(15 - c)) + 1u : 0u;
      }
    }
    sort8_desc(key);
    sort8_desc(key + 8);
#pragma unroll
    for (int i = 0; i < 8; ++i) key[i] = key[i] > key[15 - i] ? key[i] : key[15 - i];
#pragma unroll
    for (int j = 4; j > 0; j >>= 1)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if ((i & j) == 0) {
          const uint32_t x = key[i], y = key[i + j];
          key[i] = x > y ? x : y;
          key[i + j] = x > y ? y : x;
        }
    // rank j: factor H + 1 (0 past the R ranks) and codeword
    uint32_t f[8], z[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool ok = j < R && key[j] != 0u;
      f[j] = ok ? ((key[j] - 1u) >> 4) + 1u : 0u;
      z[j] = 15u - ((key[j] - 1u) & 15u);
    }
    const int shift = 4 * (G - 1 - g);
    if (g == 0) {
      // one prefix (the empty tuple): the ranks themselves
      nb = S < R ? S : R;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool ok = i < nb;
        pp[i] = pt_from<P>(ok ? f[i] : 0u);
        pc[i] = ok ? z[i] << shift : 0xFFFFFFFFu;
      }
      continue;
    }
    // candidate (i, j): product pp[i] f[j] (0 when either is absent),
    // tuple pc[i] | z[j] << shift
    auto cand = [&](int i, int j, P& cp, uint32_t& cc) {
      const bool ok = i < nb && j < R;
      cp = ok ? pt_mul(pp[i], f[j]) : pt_from<P>(0u);
      cc = ok ? (pc[i] | (z[j] << shift)) : 0xFFFFFFFFu;
    };
    P rp[8];
    uint32_t rc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) cand(i, 0, rp[i], rc[i]);
    {
      P lp[4];
      uint32_t lc[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) cand(i, 1, lp[i], lc[i]);
      merge_top8<4>(rp, rc, lp, lc);
    }
    {
      // columns 2 and 3 (prefixes 0, 1 each) merged into one sorted list
      P lp[4];
      uint32_t lc[4];
      cand(0, 2, lp[0], lc[0]);
      cand(1, 2, lp[1], lc[1]);
      cand(1, 3, lp[2], lc[2]);
      cand(0, 3, lp[3], lc[3]);
      cx_rank(lp[0], lc[0], lp[2], lc[2]);
      cx_rank(lp[1], lc[1], lp[3], lc[3]);
      cx_rank(lp[0], lc[0], lp[1], lc[1]);
      cx_rank(lp[2], lc[2], lp[3], lc[3]);
      merge_top8<4>(rp, rc, lp, lc);
    }
    {
      P lp[4];
      uint32_t lc[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) cand(0, 4 + j, lp[j], lc[j]);
      merge_top8<4>(rp, rc, lp, lc);
    }
    const int nout = S < nb * R ? S : nb * R;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bool ok = i < nout;
      pp[i] = ok ? rp[i] : pt_from<P>(0u);
      pc[i] = ok ? rc[i] : 0xFFFFFFFFu;
    }
    nb = nout;
  }
  if (mine) {
#pragma unroll
    for (int o = 0; o < 8; ++o)
      if (o < S) out[o] = o < nb ? pc[o] : 0u;
    out[SMAX] = 0u;
  }
}

// One lane per (slot, K/V) beam, 64 beams (32 slots) per wave, S <= 8.  With
// `centres` (rows formed by the readout) it also writes each slot's bias,
// tau_k into the key record's spare word and n into the value record's.
__global__ __launch_bounds__(256) void k_decode1(Dims dm, Workspace ws, int sid, int n_active, int centres) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int beam0 = (blockIdx.x * 4 + wave) * 64;
  const int beam = beam0 + lane;  // (unit * n_active + slot) * 2 + K/V
  const int nbeams = dm.units * n_active * 2;
  if (beam0 >= nbeams) return;  // uniform
  const bool bvalid = beam < nbeams;
  const int kv = beam & 1, up = bvalid ? beam >> 1 : 0;
  const int u = up / n_active, p = up % n_active;
  const size_t unit = (size_t)sid * dm.units + u;
  const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  uint32_t* out = ws.pcodes + (((size_t)u * dm.K + p) * 2 + kv) * PCW;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0;
  const int S = dm.S, C = dm.C;
  const bool nores = !pq || m.n_res == 0;
  if (bvalid && nores) out[SMAX] = 1u;
  if (centres && bvalid) {  // centres: uniform
    if (kv == 0) {
      const bool mb = (dm.flags & PROTOKV_FLAG_MASS_BIAS) != 0;
      ws.pbias[(size_t)u * dm.K + p] = mb ? logf((float)m.n) : 0.f;
      // tau_k in the key record's spare word: the readout rotates the
      // slot's formed pseudo-keys at it
      out[SMAX + 1] = (uint32_t)m.tau;
    } else {
      // n in the value record's spare word: the readout divides the slot's
      // sums by it
      out[SMAX + 1] = m.n;
    }
  }
  const bool mine = bvalid && !nores && m.n_res <= 65534u && S <= 8;
  const uint32_t* hist = reinterpret_cast<const uint32_t*>(row + (kv ? ROW_HV : ROW_HK));
  // every product the merge forms is at most prod_g max_c (H[g][c] + 1);
  // when that fits in 64 bits for all of the wave's beams the merge runs on
  // 64-bit products
  bool fits = true;
  if (mine) {
    uint64_t bound = 1;
    bool ovf = false;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint32_t mx = 0;
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4) {
        const uint4 h4 = reinterpret_cast<const uint4*>(hist + g * CMAX)[v4];
        mx = max(mx, max(max(h4.x, h4.y), max(h4.z, h4.w)));
      }
      ovf |= __builtin_mul_overflow(bound, (uint64_t)mx + 1u, &bound);
    }
    fits = !ovf;
  }
  if (__all(fits))
    decode_beam1<uint64_t>(hist, mine, S, C, out);
  else
    decode_beam1<U128>(hist, mine, S, C, out);
}

// Decoding, wide path (prototypes with more than 65534 residuals, whose
// products need 192 bits): one thread per (slot, K/V) of one (layer, kv
// head), 32 slots per
// workgroup (lanes 0-31 keys, 32-63 values).  Codes go to ws.pcodes
// [units][K][2][SMAX] (packed tuples, subspace 0 in the top nibble) and a flag
// word per (slot, K/V): 1 if the slot has no residual statistics.
template <int SM>
__global__ __launch_bounds__(64) void k_decode(Dims dm, Workspace ws, int sid, int n_active, int blocks_per_unit) {
  extern __shared__ __attribute__((aligned(16))) uint8_t s_dyn[];
  const int lane = threadIdx.x;
  const int u = blockIdx.x / blocks_per_unit;
  const int p = (blockIdx.x % blocks_per_unit) * SYN_P + (lane & 31);
  const int kv = lane >> 5;
  if (p >= n_active) return;
  const size_t unit = (size_t)sid * dm.units + u;
  const int S = dm.S;
  const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  uint32_t* out = ws.pcodes + (((size_t)u * dm.K + p) * 2 + kv) * PCW;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0;
  if (!pq || m.n_res == 0) return;             // flagged by k_decode4
  if (m.n_res <= 65534u && S <= SM) return;    // decoded by k_decode4
  out[SMAX] = 0u;
  const uint32_t* hist = reinterpret_cast<const uint32_t*>(row + (kv ? ROW_HV : ROW_HK));
  uint32_t codes[SMAX];
  {
    BeamView bv;
    bv.S = S;
    bv.w0 = reinterpret_cast<uint64_t*>(s_dyn);
    bv.w1 = bv.w0 + 2 * S * 64;
    bv.w2 = bv.w1 + 2 * S * 64;
    bv.code = reinterpret_cast<uint32_t*>(bv.w2 + 2 * S * 64);
    decode_top_s(hist, dm.C, S, bv, lane, codes);
  }
  for (int s2 = 0; s2 < S; ++s2) out[s2] = codes[s2];
}

// Pseudo-tokens: one wave per slot, lane l writes components 2l, 2l+1 of each
// of the 2S rows: k~_s = kv_dtype(float32(c + r^K_s)), v~_s likewise, with
// c = float32(sum / n) (EMA centres: the stored c) and r_s = concatenated
// codewords; bias = log n.
template <int FP32>
__global__ __launch_bounds__(256) void k_materialize(Dims dm, Workspace ws, int sid, int n_active) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int u = gw / dm.K, p = gw % dm.K;
  if (u >= dm.units || p >= n_active) return;
  const size_t unit = (size_t)sid * dm.units + u;
  // S_k rows from row rb of the unit (variance-aware allocation), else S from p S
  const bool var = ws.ps_count != nullptr;
  const int S = var ? ws.ps_count[(size_t)u * dm.K + p] : dm.S;
  const size_t rb = var ? (size_t)ws.ps_off[(size_t)u * dm.K + p] : (size_t)p * dm.S;
  const size_t es = FP32 ? 4 : 2;
  const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
  const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
  const float nf = (float)m.n;
  const float2 sk = reinterpret_cast<const float2*>(row + ROW_SUMK)[lane];
  const float2 sv = reinterpret_cast<const float2*>(row + ROW_SUMV)[lane];
  const float* cbk = ws.codebooks + unit * (2 * G * CMAX * DP);
  const int g = lane >> 3, u16 = (2 * lane) & 15;
  // rotary positions: the pseudo-keys turn at tau_k; lane l holds dims 2l,
  // 2l + 1, pair index 2 (l % 32) + {0, 1}, its partner in lane l ^ 32
  const bool rope = ws.rope_inv != nullptr;
  float rc[2] = {1.f, 1.f}, rs[2] = {0.f, 0.f};
  if (rope)
    for (int e = 0; e < 2; ++e) rope_cs((double)m.tau, ws.rope_inv[2 * (lane & 31) + e], rc[e], rs[e]);
  {
    const bool mb = (dm.flags & PROTOKV_FLAG_MASS_BIAS) != 0;
    const float bias = mb ? logf(nf) : 0.f;
    if (lane == 0) ws.pbias[(size_t)u * dm.K + p] = bias;
    if (var && lane < S) ws.prow_bias[(size_t)u * dm.K * dm.S + rb + lane] = bias;
  }
  // the decoded tuples of K and V first (all loads in flight together)
  const uint32_t* codes_k = ws.pcodes + (((size_t)u * dm.K + p) * 2) * PCW;
  const uint32_t* codes_v = codes_k + PCW;
  uint32_t ck[SMAX], cv[SMAX];
#pragma unroll
  for (int s2 = 0; s2 < SMAX; ++s2) {
    ck[s2] = s2 < S ? codes_k[s2] : 0u;
    cv[s2] = s2 < S ? codes_v[s2] : 0u;
  }
  const bool nores_k = codes_k[SMAX] != 0u, nores_v = codes_v[SMAX] != 0u;
  const int sh = 4 * (G - 1 - g);
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const float cd = (dm.flags & PROTOKV_FLAG_EMA_CENTRES) ? 1.f : nf;  // EMA centres are stored
    const float2 c = w ? make_float2(sv.x / cd, sv.y / cd) : make_float2(sk.x / cd, sk.y / cd);
    const bool nores = w ? nores_v : nores_k;
    const float* cbw = cbk + ((size_t)w * G + g) * CMAX * DP + u16;
    uint8_t* out = (w ? ws.pv : ws.pk) + ((size_t)u * dm.K * dm.S + rb) * D * es;
#pragma unroll
    for (int s2 = 0; s2 < SMAX; ++s2) {
      if (s2 < S) {
        float2 val = c;
        if (!nores) {
          const int z = ((w ? cv[s2] : ck[s2]) >> sh) & 15;
          const float2 cw = *reinterpret_cast<const float2*>(cbw + z * DP);
          val.x = c.x + cw.x;
          val.y = c.y + cw.y;
        }
        if (rope && w == 0) {  // rotate the key as rounded to the KV dtype
          if (!FP32) {
            val.x = q_from_bf16(q_to_bf16(val.x));
            val.y = q_from_bf16(q_to_bf16(val.y));
          }
          const float px = __shfl_xor(val.x, 32, 64), py = __shfl_xor(val.y, 32, 64);
          float lo, hi;
          if (lane < 32) {
            rope_pair(val.x, px, rc[0], rs[0], lo, hi);
            val.x = lo;
            rope_pair(val.y, py, rc[1], rs[1], lo, hi);
            val.y = lo;
          } else {
            rope_pair(px, val.x, rc[0], rs[0], lo, hi);
            val.x = hi;
            rope_pair(py, val.y, rc[1], rs[1], lo, hi);
            val.y = hi;
          }
        }
        if (FP32) {
          reinterpret_cast<float2*>(out + (size_t)s2 * D * 4)[lane] = val;
        } else {
          const uint32_t packed = (uint32_t)q_to_bf16(val.x) | ((uint32_t)q_to_bf16(val.y) << 16);
          reinterpret_cast<uint32_t*>(out + (size_t)s2 * D * 2)[lane] = packed;
        }
      }
    }
  }
}

// bf16 pseudo-tokens, one wave per slot with 16-byte stores: lane l writes
// dims [8 (l % 16), 8 (l % 16) + 8) of rows s = l / 16 + 4 i (i = 0, 1, ...)
// of K and of V, so each store instruction covers four whole rows.  The
// values and their rounding are those of k_materialize.
__global__ __launch_bounds__(256) void k_materialize16(Dims dm, Workspace ws, int sid, int n_active) {
  const int lane = threadIdx.x & 63;
  const int gw = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int u = gw / dm.K, p = gw % dm.K;
  if (u >= dm.units || p >= n_active) return;
  const size_t unit = (size_t)sid * dm.units + u;
  // S_k rows from row rb of the unit (variance-aware allocation), else S from p S
  const bool var = ws.ps_count != nullptr;
  const int S = var ? ws.ps_count[(size_t)u * dm.K + p] : dm.S;
  const size_t rb = var ? (size_t)ws.ps_off[(size_t)u * dm.K + p] : (size_t)p * dm.S;
  const int dq = lane & 15, r0 = lane >> 4;
  const int g = dq >> 1, hsub = (dq & 1) * 8;  // subspace of these 8 dims, offset inside it
  const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
  const float nf = (float)reinterpret_cast<const RowMeta*>(row + ROW_META)->n;
  const uint32_t* codes = ws.pcodes + (((size_t)u * dm.K + p) * 2) * PCW;
  // rotary positions: the pseudo-keys turn at tau_k; this lane's dims are
  // pair indices 8 (dq % 8) + e, the partners in lane dq ^ 8
  const bool rope = ws.rope_inv != nullptr;
  float rc[8], rs[8];
  if (rope) {
    const double tau = (double)reinterpret_cast<const RowMeta*>(row + ROW_META)->tau;
#pragma unroll
    for (int e = 0; e < 8; ++e) rope_cs(tau, ws.rope_inv[8 * (dq & 7) + e], rc[e], rs[e]);
  }
  const float* cbk = ws.codebooks + unit * (2 * G * CMAX * DP);
  {
    const bool mb = (dm.flags & PROTOKV_FLAG_MASS_BIAS) != 0;
    const float bias = mb ? logf(nf) : 0.f;
    if (lane == 0) ws.pbias[(size_t)u * dm.K + p] = bias;
    if (var && lane < S) ws.prow_bias[(size_t)u * dm.K * dm.S + rb + lane] = bias;
  }
  // everything this lane needs first: its 8 dims of both sums, the no-residual
  // flags and the tuples of its rows
  float4 sr[2][2];
  uint32_t tup[2][SMAX / 4];
  bool nores[2];
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const float* sums = reinterpret_cast<const float*>(row + (w ? ROW_SUMV : ROW_SUMK)) + 8 * dq;
    sr[w][0] = reinterpret_cast<const float4*>(sums)[0];
    sr[w][1] = reinterpret_cast<const float4*>(sums)[1];
    const uint32_t* cw = codes + w * PCW;
    nores[w] = cw[SMAX] != 0u;
#pragma unroll
    for (int i = 0; i < SMAX / 4; ++i) {
      const int s2 = r0 + 4 * i;
      tup[w][i] = s2 < S ? cw[s2] : 0u;
    }
  }
  const int sh = 4 * (G - 1 - g);
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const float cd = (dm.flags & PROTOKV_FLAG_EMA_CENTRES) ? 1.f : nf;  // EMA centres are stored
    const float c[8] = {sr[w][0].x / cd, sr[w][0].y / cd, sr[w][0].z / cd, sr[w][0].w / cd,
                        sr[w][1].x / cd, sr[w][1].y / cd, sr[w][1].z / cd, sr[w][1].w / cd};
    const float* cbw = cbk + ((size_t)w * G + g) * CMAX * DP + hsub;
    uint8_t* out = (w ? ws.pv : ws.pk) + ((size_t)u * dm.K * dm.S + rb) * D * 2 + dq * 16;
#pragma unroll
    for (int i = 0; i < SMAX / 4; ++i) {
      const int s2 = r0 + 4 * i;
      if (s2 < S) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = c[e];
        if (!nores[w]) {
          const int z = (tup[w][i] >> sh) & 15;
          const float4 a = reinterpret_cast<const float4*>(cbw + z * DP)[0];
          const float4 b = reinterpret_cast<const float4*>(cbw + z * DP)[1];
          v[0] = c[0] + a.x; v[1] = c[1] + a.y; v[2] = c[2] + a.z; v[3] = c[3] + a.w;
          v[4] = c[4] + b.x; v[5] = c[5] + b.y; v[6] = c[6] + b.z; v[7] = c[7] + b.w;
        }
        if (rope && w == 0) {  // rotate the key as rounded to bf16
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = q_from_bf16(q_to_bf16(v[e]));
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float pv = __shfl_xor(v[e], 8, 64);
            float lo, hi;
            if (dq < 8) {
              rope_pair(v[e], pv, rc[e], rs[e], lo, hi);
              v[e] = lo;
            } else {
              rope_pair(pv, v[e], rc[e], rs[e], lo, hi);
              v[e] = hi;
            }
          }
        }
        uint4 o;
        o.x = (uint32_t)q_to_bf16(v[0]) | ((uint32_t)q_to_bf16(v[1]) << 16);
        o.y = (uint32_t)q_to_bf16(v[2]) | ((uint32_t)q_to_bf16(v[3]) << 16);
        o.z = (uint32_t)q_to_bf16(v[4]) | ((uint32_t)q_to_bf16(v[5]) << 16);
        o.w = (uint32_t)q_to_bf16(v[6]) | ((uint32_t)q_to_bf16(v[7]) << 16);
        *reinterpret_cast<uint4*>(out + (size_t)s2 * D * 2) = o;
      }
    }
  }
}

hipError_t launch_decode(const Dims& dm, const Workspace& ws, int sid, int n_active, bool centres, bool wide,
                         hipStream_t st) {
  if (n_active <= 0) return hipSuccess;
  const int bpu = (n_active + SYN_P - 1) / SYN_P;
  const size_t lds = (size_t)2 * dm.S * 64 * (3 * sizeof(uint64_t) + sizeof(uint32_t));
  const int nbeams = dm.units * n_active * 2;
  constexpr int LPB = 2;  // lanes per beam
  const int nblk = (nbeams + 4 * (64 / LPB) - 1) / (4 * (64 / LPB));
  if (dm.S <= 8) {
    const int nblk1 = (nbeams + 255) / 256;
    hipLaunchKernelGGL(k_decode1, dim3(nblk1), dim3(256), 0, st, dm, ws, sid, n_active, centres ? 1 : 0);
    if (wide) hipLaunchKernelGGL(k_decode<8>, dim3(dm.units * bpu), dim3(64), lds, st, dm, ws, sid, n_active, bpu);
  } else {
    hipLaunchKernelGGL((k_decode4<16, LPB>), dim3(nblk), dim3(256), 0, st, dm, ws, sid, n_active, centres ? 1 : 0);
    if (wide) hipLaunchKernelGGL(k_decode<16>, dim3(dm.units * bpu), dim3(64), lds, st, dm, ws, sid, n_active, bpu);
  }
  return hipGetLastError();
}

// Eight consecutive KV elements at element offset e of `base` as float, and back.
template <int FP32>
__device__ __forceinline__ void ld8kv(const uint8_t* base, size_t e, float (&x)[8]) {
  if (FP32) {
    const float4 a = reinterpret_cast<const float4*>(base + e * 4)[0];
    const float4 b = reinterpret_cast<const float4*>(base + e * 4)[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  } else {
    const uint4 w = *reinterpret_cast<const uint4*>(base + e * 2);
    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = __uint_as_float(ww[q] << 16);
      x[2 * q + 1] = __uint_as_float(ww[q] & 0xFFFF0000u);
    }
  }
}
template <int FP32>
__device__ __forceinline__ void st8kv(uint8_t* base, size_t e, const float (&x)[8]) {
  if (FP32) {
    reinterpret_cast<float4*>(base + e * 4)[0] = make_float4(x[0], x[1], x[2], x[3]);
    reinterpret_cast<float4*>(base + e * 4)[1] = make_float4(x[4], x[5], x[6], x[7]);
  } else {
    uint4 o;
    o.x = (uint32_t)q_to_bf16(x[0]) | ((uint32_t)q_to_bf16(x[1]) << 16);
    o.y = (uint32_t)q_to_bf16(x[2]) | ((uint32_t)q_to_bf16(x[3]) << 16);
    o.z = (uint32_t)q_to_bf16(x[4]) | ((uint32_t)q_to_bf16(x[5]) << 16);
    o.w = (uint32_t)q_to_bf16(x[6]) | ((uint32_t)q_to_bf16(x[7]) << 16);
    *reinterpret_cast<uint4*>(base + e * 2) = o;
  }
}

// Rotates the rows of one token vector: pair indices [8 c, 8 c + 8) (dims
// 8c.. and D/2 + 8c..) of the row at element offset `e0`, at position pos.
template <int FP32>
__device__ __forceinline__ void rope_row8(const uint8_t* src, uint8_t* dst, size_t e0, int c, double pos,
                                          const double* inv) {
  float x1[8], x2[8], y1[8], y2[8];
  ld8kv<FP32>(src, e0 + 8 * c, x1);
  ld8kv<FP32>(src, e0 + D / 2 + 8 * c, x2);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float cs, sn;
    rope_cs(pos, inv[8 * c + e], cs, sn);
    rope_pair(x1[e], x2[e], cs, sn, y1[e], y2[e]);
  }
  st8kv<FP32>(dst, e0 + 8 * c, y1);
  st8kv<FP32>(dst, e0 + D / 2 + 8 * c, y2);
}

// The query [L][tq][Hq][D] rotated into qrot: thread = (row, pair block c);
// token t at position p0 + t.
template <int FP32>
__global__ __launch_bounds__(256) void k_rope_q(Dims dm, Workspace ws, const uint8_t* q, int tq, long long p0) {
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t row = gid >> 3;
  if (row >= (size_t)dm.L * tq * dm.Hq) return;
  const int c = (int)(gid & 7);
  const int t = (int)((row / dm.Hq) % tq);
  rope_row8<FP32>(q, ws.qrot, row * D, c, (double)(p0 + t), ws.rope_inv);
}

// Ring insert with rotary positions, in one pass: thread = (entry, unit,
// token j, pair block c) copies the token's K and V chunks [8c, 8c + 8) and
// [D/2 + 8c, D/2 + 8c + 8) into the ring and writes the K pair rotated at
// its stream position f * T + j into ring_kr.
template <int FP32>
__global__ __launch_bounds__(256) void k_ring_insert_rope(Dims dm, Workspace ws, AppendBatch ab,
                                                          const uint8_t* k, const uint8_t* v) {
  const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
  const size_t per = (size_t)dm.units * dm.T * 8;
  const int e = (int)(gid / per);
  if (e >= ab.n) return;
  const size_t r = gid % per;
  const int c = (int)(r & 7), j = (int)((r >> 3) % dm.T), u = (int)((r >> 3) / dm.T);
  const size_t es = FP32 ? 4 : 2;
  const size_t s0 = (((size_t)e * dm.units + u) * dm.T + j) * (size_t)D;
  const size_t d0 = ((((size_t)ab.sid[e] * dm.units + u) * (dm.W + 1) + ab.slot[e]) * dm.T + j) * (size_t)D;
  constexpr int W16 = FP32 ? 2 : 1;  // 16-byte words per 8 elements
  uint4 ka[W16], kb[W16], va[W16], vb[W16];
#pragma unroll
  for (int w = 0; w < W16; ++w) {
    ka[w] = reinterpret_cast<const uint4*>(k + (s0 + 8 * c) * es)[w];
    kb[w] = reinterpret_cast<const uint4*>(k + (s0 + D / 2 + 8 * c) * es)[w];
    va[w] = reinterpret_cast<const uint4*>(v + (s0 + 8 * c) * es)[w];
    vb[w] = reinterpret_cast<const uint4*>(v + (s0 + D / 2 + 8 * c) * es)[w];
  }
#pragma unroll
  for (int w = 0; w < W16; ++w) {
    reinterpret_cast<uint4*>(ws.ring_k + (d0 + 8 * c) * es)[w] = ka[w];
    reinterpret_cast<uint4*>(ws.ring_k + (d0 + D / 2 + 8 * c) * es)[w] = kb[w];
    reinterpret_cast<uint4*>(ws.ring_v + (d0 + 8 * c) * es)[w] = va[w];
    reinterpret_cast<uint4*>(ws.ring_v + (d0 + D / 2 + 8 * c) * es)[w] = vb[w];
  }
  float x1[8], x2[8], y1[8], y2[8];
  ld8kv<FP32>(reinterpret_cast<const uint8_t*>(ka), 0, x1);
  ld8kv<FP32>(reinterpret_cast<const uint8_t*>(kb), 0, x2);
  const double pos = (double)ab.frame[e] * dm.T + j;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    float cs, sn;
    rope_cs(pos, ws.rope_inv[8 * c + q], cs, sn);
    rope_pair(x1[q], x2[q], cs, sn, y1[q], y2[q]);
  }
  st8kv<FP32>(ws.ring_kr, d0 + 8 * c, y1);
  st8kv<FP32>(ws.ring_kr, d0 + D / 2 + 8 * c, y2);
}

hipError_t launch_ring_insert_rope(const Dims& dm, const Workspace& ws, const AppendBatch& ab, const void* k,
                                   const void* v, hipStream_t st) {
  const size_t n = (size_t)ab.n * dm.units * dm.T * 8;
  const dim3 grid((unsigned)((n + 255) / 256));
  const uint8_t* kb = static_cast<const uint8_t*>(k);
  const uint8_t* vb = static_cast<const uint8_t*>(v);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_ring_insert_rope<1>, grid, dim3(256), 0, st, dm, ws, ab, kb, vb);
  else
    hipLaunchKernelGGL(k_ring_insert_rope<0>, grid, dim3(256), 0, st, dm, ws, ab, kb, vb);
  return hipGetLastError();
}

hipError_t launch_rope_q(const Dims& dm, const Workspace& ws, const void* q, int tq, long long p0,
                         hipStream_t st) {
  const size_t n = (size_t)dm.L * tq * dm.Hq * 8;
  const dim3 grid((unsigned)((n + 255) / 256));
  const uint8_t* qb = static_cast<const uint8_t*>(q);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_rope_q<1>, grid, dim3(256), 0, st, dm, ws, qb, tq, p0);
  else
    hipLaunchKernelGGL(k_rope_q<0>, grid, dim3(256), 0, st, dm, ws, qb, tq, p0);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Variance-aware pseudo-token counts (appendix "Dynamic Pseudo-Token
// Allocation").  Workgroup = one (layer, kv head) of stream sid.  Every
// thread computes Var(H_k) of its slots in float64, in the order the
// definition sums (sides, subspaces, codewords, dims ascending); one thread
// takes the sums over slots in slot order (water-filling of the shares over
// the cap, then cumulative rounding), the others compute the shares.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_alloc(Dims dm, Workspace ws, int sid, int A) {
  __shared__ double s_var[AL_KMAX];
  __shared__ double s_x[AL_KMAX];
  __shared__ uint8_t s_cap[AL_KMAX];
  __shared__ float s_cb[2 * G * CMAX * DP];
  __shared__ double s_n2[2 * G * CMAX];
  __shared__ double s_par[2];   // remaining budget, variance sum of the uncapped
  __shared__ int s_flag;
  const int tid = threadIdx.x, u = blockIdx.x;
  const size_t unit = (size_t)sid * dm.units + u;
  const int C = dm.C, S = dm.S, smax = dm.pseudo_max;
  const float* cbk = ws.codebooks + unit * (2 * G * CMAX * DP);
  for (int i = tid; i < 2 * G * CMAX * DP; i += 256) s_cb[i] = cbk[i];
  __syncthreads();
  if (tid < 2 * G * CMAX) {
    double n2 = 0.0;
    for (int d = 0; d < DP; ++d) {
      const double c = (double)s_cb[tid * DP + d];
      n2 = n2 + c * c;
    }
    s_n2[tid] = n2;
  }
  __syncthreads();
  for (int k = tid; k < A; k += 256) {
    const uint8_t* row = ws.bank + (unit * dm.K + k) * ROW;
    const uint32_t nres = reinterpret_cast<const RowMeta*>(row + ROW_META)->n_res;
    double total = 0.0;
    if (nres > 0) {
      const double den = (double)nres;
      for (int side = 0; side < 2; ++side) {
        const uint32_t* hist = reinterpret_cast<const uint32_t*>(row + (side ? ROW_HV : ROW_HK));
        for (int g = 0; g < G; ++g) {
          double e2 = 0.0, mean[DP];
#pragma unroll
          for (int d = 0; d < DP; ++d) mean[d] = 0.0;
          for (int c = 0; c < C; ++c) {
            const double pc = (double)hist[g * CMAX + c] / den;
            e2 = e2 + pc * s_n2[(side * G + g) * CMAX + c];
            const float* cw = s_cb + ((side * G + g) * CMAX + c) * DP;
#pragma unroll
            for (int d = 0; d < DP; ++d) mean[d] = mean[d] + pc * (double)cw[d];
          }
          double m2 = 0.0;
#pragma unroll
          for (int d = 0; d < DP; ++d) m2 = m2 + mean[d] * mean[d];
          const double v = e2 - m2;
          total = total + (v > 0.0 ? v : 0.0);
        }
      }
    }
    s_var[k] = total;
    s_cap[k] = 0;
  }
  __syncthreads();
  const int tot = A * S;
  __shared__ int s_novar;
  if (tid == 0) {
    double w = 0.0;
    for (int k = 0; k < A; ++k) w += s_var[k];
    s_novar = w == 0.0 ? 1 : 0;  // no variance at all: every S_k = S
  }
  __syncthreads();
  if (!s_novar) {
    int ncap = 0;
    for (;;) {  // uniform: every thread sees the same ncap and flags
      if (tid == 0) {
        double w = 0.0;
        for (int k = 0; k < A; ++k)
          if (!s_cap[k]) w += s_var[k];
        s_par[0] = (double)(tot - A - ncap * (smax - 1));
        s_par[1] = w;
        s_flag = 0;
      }
      __syncthreads();
      const double rest = s_par[0], w = s_par[1];
      const double nunc = (double)(A - ncap);
      for (int k = tid; k < A; k += 256) {
        double x;
        if (s_cap[k]) x = (double)smax;
        else if (w > 0.0) x = 1.0 + rest * s_var[k] / w;
        else x = 1.0 + rest / nunc;
        s_x[k] = x;
        if (!s_cap[k] && x > (double)smax) s_flag = 1;  // every writer stores 1
      }
      __syncthreads();
      const int again = s_flag;
      __syncthreads();
      if (!again) break;
      for (int k = tid; k < A; k += 256)
        if (!s_cap[k] && s_x[k] > (double)smax) s_cap[k] = 1;
      __syncthreads();
      if (tid == 0) {
        int n = 0;
        for (int k = 0; k < A; ++k) n += s_cap[k];
        s_par[0] = (double)n;
      }
      __syncthreads();
      ncap = (int)s_par[0];
      __syncthreads();
    }
  }
  if (tid == 0) {
    int32_t* cnt = ws.ps_count + (size_t)u * dm.K;
    int32_t* off = ws.ps_off + (size_t)u * dm.K;
    // cumulative rounding: S_k = floor(X_k + 1/2) - floor(X_(k-1) + 1/2)
    double X = 0.0;
    long long prev = 0;
    for (int k = 0; k < A; ++k) {
      off[k] = (int32_t)prev;
      if (s_novar) {
        cnt[k] = S;
        prev += S;
        continue;
      }
      X += s_x[k];
      const long long cur = (long long)floor(X + 0.5);
      cnt[k] = (int32_t)(cur - prev);
      prev = cur;
    }
    for (int k = A; k < dm.K; ++k) {
      cnt[k] = 0;
      off[k] = (int32_t)prev;
    }
  }
}

hipError_t launch_alloc(const Dims& dm, const Workspace& ws, int sid, int n_active, hipStream_t st) {
  hipLaunchKernelGGL(k_alloc, dim3(dm.units), dim3(256), 0, st, dm, ws, sid, n_active);
  return hipGetLastError();
}

hipError_t launch_materialize(const Dims& dm, const Workspace& ws, int sid, int n_active, hipStream_t st) {
  if (n_active <= 0) return hipSuccess;
  const int waves = dm.units * dm.K;
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_materialize<1>, dim3((waves + 3) / 4), dim3(256), 0, st, dm, ws, sid, n_active);
  else
    hipLaunchKernelGGL(k_materialize16, dim3((waves + 3) / 4), dim3(256), 0, st, dm, ws, sid, n_active);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Readout.  Context of kv head u: near tokens (frames f_first.. in ring
// slots f mod (W+1)), then pseudo-tokens; logit = q.k/sqrt(D) + bias with
// bias 0 on near tokens and log n_k on the pseudo-tokens of slot k.
// Query rows of one kv head: r = t * (Hq/Hkv) + g  (query head u_h*grp + g).
// ---------------------------------------------------------------------------
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

struct CtxRef {
  const uint8_t* base;
  float bias;
  bool ok;
};

template <int ES>
__device__ __forceinline__ CtxRef ctx_key(const Dims& dm, const Workspace& ws, const AttendArgs& aa,
                                          size_t unit, int u, int idx, bool values) {
  CtxRef r;
  r.ok = idx < aa.n_near + aa.n_far;
  r.bias = 0.f;
  if (!r.ok) { r.base = nullptr; return r; }
  if (idx < aa.n_near) {
    const int f = aa.f_first + idx / dm.T;
    const int tok = idx - (idx / dm.T) * dm.T;
    const int slot = f % (dm.W + 1);
    r.base = (values ? ws.ring_v : aa.near_k) + (((unit * (dm.W + 1) + slot) * dm.T + tok) * (size_t)D) * ES;
  } else {
    const int row = idx - aa.n_near;
    r.base = (values ? ws.pv : ws.pk) + (((size_t)u * dm.K * dm.S + row) * (size_t)D) * ES;
    r.bias = aa.rowbias ? aa.rowbias[(size_t)u * dm.K * dm.S + row] : ws.pbias[(size_t)u * dm.K + row / dm.S];
  }
  return r;
}

// bf16 path.  Workgroup = eight waves for one (kv head, context split,
// block of query rows): one wave per 32 rows for up to 256 rows (KH = 1), or
// for at most 128 rows two waves per 32 rows, each taking one 32-key half
// of every tile, their results merged at the end (KH = 2), so each SIMD
// runs two waves either way.  A context tile of 64
// keys sits in LDS in two layouts under which every operand read is a per-lane
// base plus compile-time offsets and touches distinct banks:
//   K chunk-major: 16-byte chunk c (dims 8c .. 8c+7) of row r at c * 1024 + r * 16;
//   V by 32-dim block: dims 32b .. 32b+31 of row r at b * 4096 + r * 64.
// Near-window tiles go straight from global memory into these layouts
// (global_load_lds_dwordx4), three tiles ahead of the one computed.
// S^T = K Q^T and O^T = V^T P with v_mfma_f32_32x32x16_bf16; the V^T operand
// comes through ds_read_b64_tr_b16.  Each lane holds one query column, so the
// online softmax is lane-local plus one exchange with the partner lane.  With
// several splits, every workgroup writes its partial (unnormalised O, running
// max, sum) for k_attend_merge.
constexpr int AT_KEYS = 64;
constexpr int AT_ROWS = 256;  // query rows per workgroup
constexpr int AT_TILE_BYTES = AT_KEYS * D * 2;   // one K or V tile, 16 KB

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void gbl_void;

// Barrier for LDS traffic only: waits for this wave's LDS operations, not
// for its outstanding global loads (the tiles in flight).  The asm memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  asm volatile("s_barrier" ::: "memory");
}
constexpr int AT_NBUF = 4;        // tile buffers: tile t computes while t+1..t+3 load
constexpr int AT_NTAB = 5;        // row-table entries (written 3 tiles ahead)
constexpr int AT_PB_MAX = 2048;   // pseudo-token biases staged in LDS up to this capacity

template <int NW, int KH>
__global__ __launch_bounds__(NW * 64, 1) void k_attend_bf16(Dims dm, Workspace ws, AttendArgs aa, int rows, int rblocks) {
  constexpr int LPT = 32 / NW;  // load instructions per wave per tile
  constexpr int RPW = NW * 32 / KH;  // query rows per workgroup
  __shared__ __attribute__((aligned(16))) uint8_t s_kv[AT_NBUF][2][AT_TILE_BYTES];   // [buffer][K,V]
  __shared__ __attribute__((aligned(16))) float s_bias[AT_NTAB][AT_KEYS];           // log2(e) * bias, -inf past the context
  __shared__ const uint8_t* s_rowp[AT_NTAB][2][AT_KEYS];                             // K and V address of each tile row
  __shared__ float s_pb[AT_PB_MAX];                                                  // log2(e) * ln n_k of this unit
  // rotary positions: (cos, sin) of tau_k * theta^(-2i/D) for the slots of
  // a formed tile, two tiles' tables (the next one's is written ahead)
  __shared__ float2 s_rtab[2][PS_SLOTS][D / 2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // blocks of one kv head land on one XCD (dispatch is round-robin over 8)
  const int nblk = gridDim.x, per = nblk / 8;
  const int lbid = (int)blockIdx.x < per * 8 ? ((int)blockIdx.x % 8) * per + (int)blockIdx.x / 8 : (int)blockIdx.x;
  const int split = lbid % aa.splits;
  const int rb = (lbid / aa.splits) % rblocks;
  const int u = lbid / (aa.splits * rblocks);
  const size_t unit = (size_t)aa.sid * dm.units + u;
  const int grp = dm.Hq / dm.Hkv;
  const int l = u / dm.Hkv, kvh = u % dm.Hkv;
  const int ctx = aa.n_near + aa.n_far;
  // rows [c0, c1n) stream through LDS by DMA: with aa.gen the split's share
  // of the near window (the pseudo-token rows [ps0, ps1) of its share are
  // formed in LDS from the synthesized centres, decode records and
  // codebooks), else context rows [c0, c1) of the near window followed by
  // the written pseudo-token rows
  const int c0 = aa.gen ? min(aa.n_near, split * aa.near_chunk) : split * aa.chunk;
  const int c1n = aa.gen ? min(aa.n_near, c0 + aa.near_chunk) : min(ctx, c0 + aa.chunk);
  const int ntiles = c1n > c0 ? (c1n - c0 + AT_KEYS - 1) / AT_KEYS : 0;
  const bool pb_lds = dm.K <= AT_PB_MAX;
  if (pb_lds)
    for (int k = tid; k < dm.K; k += NW * 64) s_pb[k] = ws.pbias[(size_t)u * dm.K + k] * LOG2E;

  const int col = lane & 31, half = lane >> 5;
  // KH = 2: waves w and w + NW / 2 take the same 32 query rows and the two
  // 32-key halves of every tile
  const int rblk = KH == 2 ? wave % (NW / 2) : wave, kh = KH == 2 ? wave / (NW / 2) : 0;
  const int r = rb * RPW + rblk * 32 + col;  // query row of this lane
  const bool rvalid = r < rows;
  const bool wvalid = rb * RPW + rblk * 32 < rows;  // uniform: the wave has query rows
  bf16x8 bq[8];
  {
    const int t = rvalid ? r / grp : 0, gg = rvalid ? r % grp : 0;
    const uint16_t* qr = reinterpret_cast<const uint16_t*>(aa.q) +
                         ((((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg) * D);
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      u16x8 v = *reinterpret_cast<const u16x8*>(qr + kk * 16 + half * 8);
      if (!rvalid) v = (u16x8)0;
      bq[kk] = __builtin_bit_cast(bf16x8, v);
    }
  }
  __syncthreads();  // s_pb staged (and the query loads complete)

  // Per-tile row table: wave 0 resolves each tile row (one lane per row) to its
  // K and V addresses and its bias once, three tiles ahead.  Rows past the
  // context read row c0 and carry bias -inf.
  const float invS = 1.0f / (float)dm.S;
  auto resolve = [&](int t, const uint8_t*& kp, const uint8_t*& vp, float& bv) {
    const int idx = c0 + t * AT_KEYS + lane;
    const int pos = idx < c1n ? idx : c0;
    bv = idx < c1n ? 0.f : -INFINITY;
    if (pos < aa.n_near) {
      const int fo = pos / dm.T;
      const int slot = (aa.f_first + fo) % (dm.W + 1);
      const size_t off = (((unit * (dm.W + 1) + slot) * dm.T + (pos - fo * dm.T)) * (size_t)D) * 2;
      kp = aa.near_k + off;
      vp = ws.ring_v + off;
    } else {
      const int prow = pos - aa.n_near;
      const size_t off = (((size_t)u * dm.K * dm.S + prow) * (size_t)D) * 2;
      kp = ws.pk + off;
      vp = ws.pv + off;
      if (aa.rowbias) {
        if (idx < c1n) bv = aa.rowbias[(size_t)u * dm.K * dm.S + prow] * LOG2E;
      } else {
        int k = (int)((float)prow * invS);
        k -= k * dm.S > prow ? 1 : 0;
        k += (k + 1) * dm.S <= prow ? 1 : 0;
        if (idx < c1n) bv = pb_lds ? s_pb[k] : ws.pbias[(size_t)u * dm.K + k] * LOG2E;
      }
    }
  };
  auto publish = [&](int t, const uint8_t* kp, const uint8_t* vp, float bv) {
    const int e = t % AT_NTAB;
    s_rowp[e][0][lane] = kp;
    s_rowp[e][1][lane] = vp;
    s_bias[e][lane] = bv;
  };
  // Loads of tile t into LDS buffer t % AT_NBUF: instruction i = wave + q * NW
  // (q < LPT) moves 1 KiB, K chunk i of all 64 rows (lane = row) for i < 16,
  // else V block j = i - 16: dims 32 (j / 4) .. +31 of rows 16 (j % 4) ..
  // +15 (lane / 4 = row, lane % 4 = 16-byte part).
  auto issue = [&](int t) {
    const int e = t % AT_NTAB, buf = t % AT_NBUF;
#pragma unroll
    for (int q = 0; q < LPT; ++q) {
      const int i = wave + q * NW;  // uniform
      const uint8_t* src;
      if (i < 16) {
        src = s_rowp[e][0][lane] + i * 16;
      } else {
        const int j = i - 16;
        src = s_rowp[e][1][(j & 3) * 16 + (lane >> 2)] + ((j >> 2) * 4 + (lane & 3)) * 16;
      }
      lds_dma16(src, &s_kv[buf][i >> 4][(i & 15) * 1024]);
    }
  };

  const float scale = LOG2E / sqrtf((float)D);
  f32x16 oacc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) oacc[b] = (f32x16){0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  // Reference max (log2 units) with a finite floor: masked keys score -inf and
  // give exp2(-inf) = 0 without special cases.  The reference is raised only
  // when a row's max exceeds it by more than 8, so p <= 2^8 and the output
  // accumulators are rescaled rarely.
  float mref = -1e30f, lrun = 0.f;

  // per-lane operand bases: K row h*32 + col, chunk 2 kk + half at
  // koff + kk * 2048 + h * 512; V (transposed reads, see below) at
  // voff + b * 4096 + st * 1024 (+ 512 for keys 8 .. 15 of the step)
  const int grp16 = lane >> 4, s16 = lane & 15;
  const int koff = half * 1024 + col * 16;
  const int voff = (4 * half + (s16 >> 2)) * 64 + (grp16 & 1) * 32 + (s16 & 3) * 8;
  const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  // one 64-key tile in LDS (K at kt, V at vt): S^T = K Q^T, scores with the
  // tile's biases, online softmax, O^T += V^T P.  Without BIAS (a full tile of
  // near-window keys after the first tile, all biases 0) the scores are taken
  // relative to the running reference in the same multiply-add.
  auto compute_tile = [&](const uint8_t* kt, const uint8_t* vt, int tb, auto bias_tag) {
    constexpr bool BIAS = decltype(bias_tag)::value;
    const uint8_t* kl = kt + koff;
    const uint8_t* vl = vt + voff;
    // S^T for the wave's 32-key halves of the tile (both, or half kh)
    constexpr int NH = 2 / KH;
    f32x16 sacc[NH];
  #pragma unroll
    for (int hh = 0; hh < NH; ++hh) {
      const int h = KH == 2 ? kh : hh;
      sacc[hh] = (f32x16){0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  #pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const bf16x8 ak = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(kl + kk * 2048 + h * 512));
        sacc[hh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak, bq[kk], sacc[hh], 0, 0, 0);
      }
    }
    // scores x = s * scale + bias (key m = h*32 + (i/4)*8 + half*4 + i%4),
    // without BIAS x = s * scale - mref
    float tmax = -1e30f;
    if constexpr (BIAS) {
  #pragma unroll
      for (int hh = 0; hh < NH; ++hh) {
        const int h = KH == 2 ? kh : hh;
  #pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const float4 bb = *reinterpret_cast<const float4*>(&s_bias[tb][h * 32 + i4 * 8 + half * 4]);
          const float bv[4] = {bb.x, bb.y, bb.z, bb.w};
  #pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = fmaf(sacc[hh][i4 * 4 + e], scale, bv[e]);
            sacc[hh][i4 * 4 + e] = x;
            tmax = fmaxf(tmax, x);
          }
        }
      }
    } else {
      const float nm = -mref;
  #pragma unroll
      for (int hh = 0; hh < NH; ++hh)
  #pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float x = fmaf(sacc[hh][i], scale, nm);
          sacc[hh][i] = x;
          tmax = fmaxf(tmax, x);
        }
    }
    tmax = fmaxf(tmax, xor32(tmax));
    // the reference moves up only when a row's max exceeds it by more than 8
    const bool grow = BIAS ? tmax > mref + 8.0f : tmax > 8.0f;
    if (__ballot(grow)) {  // uniform
      if constexpr (BIAS) {
        const float mnew = grow ? tmax : mref;
        const float alpha = __builtin_amdgcn_exp2f(mref - mnew);
        lrun *= alpha;
  #pragma unroll
        for (int b = 0; b < 4; ++b)
  #pragma unroll
          for (int i = 0; i < 16; ++i) oacc[b][i] *= alpha;
        mref = mnew;
      } else {
        const float mnew = grow ? mref + tmax : mref;
        const float delta = mnew - mref;
        const float alpha = __builtin_amdgcn_exp2f(-delta);
        lrun *= alpha;
  #pragma unroll
        for (int b = 0; b < 4; ++b)
  #pragma unroll
          for (int i = 0; i < 16; ++i) oacc[b][i] *= alpha;
  #pragma unroll
        for (int hh = 0; hh < NH; ++hh)
  #pragma unroll
          for (int i = 0; i < 16; ++i) sacc[hh][i] -= delta;
        mref = mnew;
      }
    }
    // P in bf16; the row sum is taken over the rounded values the products use
    bf16x8 pb[2 * NH];
  #pragma unroll
    for (int hh = 0; hh < NH; ++hh)
  #pragma unroll
      for (int i = 0; i < 16; ++i)
        pb[2 * hh + (i >> 3)][i & 7] = (__bf16)__builtin_amdgcn_exp2f(BIAS ? sacc[hh][i] - mref : sacc[hh][i]);
    float sum0 = 0.f, sum1 = 0.f;
  #pragma unroll
    for (int j = 0; j < 2 * NH; ++j) {
      sum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 0, 1), ones2, sum0, false);
      sum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 2, 3), ones2, sum1, false);
      sum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 4, 5), ones2, sum0, false);
      sum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[j], pb[j], 6, 7), ones2, sum1, false);
    }
    float psum = sum0 + sum1;
    psum += xor32(psum);
    lrun += psum;
    // O^T = V^T P.  k positions half*8 + i of step st <-> keys 16 st + 4 half + {0..3}
    // (i < 4) and 16 st + 8 + 4 half + {0..3} (i >= 4), matching P's layout.  Each
    // 4-key part is one ds_read_b64_tr_b16 per 16-lane group: source lane s reads
    // key key0 + s/4, dims d0 + 4(s%4) .. +3 (d0 = 32 b + 16 (lane/16 % 2)); lane i
    // then holds dim d0 + i of the 4 keys.
  #pragma unroll
    for (int b = 0; b < 4; ++b) {
  #pragma unroll
      for (int st = 0; st < 2 * NH; ++st) {
        const int sk = KH == 2 ? 2 * kh + st : st;  // 16-key step of the tile
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vl + b * 4096 + sk * 1024));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vl + b * 4096 + sk * 1024 + 512));
        const v8i16 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), pb[st], oacc[b], 0, 0, 0);
      }
    }
  };

  // prologue: rows of tiles 0..2 published, their loads issued; tile 3 resolved
  const uint8_t *nk = nullptr, *nv = nullptr;
  float nb = -INFINITY;
  if (wave == 0) {
    for (int t = 0; t < 3 && t < ntiles; ++t) {
      resolve(t, nk, nv, nb);
      publish(t, nk, nv, nb);
    }
    if (ntiles > 3) resolve(3, nk, nv, nb);
  }
  wait_vm<0>();  // the query operands are in registers before any tile is in flight
  lds_barrier();
  for (int t = 0; t < 3 && t < ntiles; ++t) issue(t);

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t % AT_NBUF, tb = t % AT_NTAB;
    // this wave's loads of tile t have landed; tiles t+1, t+2 may still be in flight
    if (t + 2 < ntiles) wait_vm<2 * LPT>();
    else if (t + 1 < ntiles) wait_vm<LPT>();
    else wait_vm<0>();
    // entry (t + 3) % 5 was last read for tile t - 2 (before the previous barrier)
    if (wave == 0 && t + 3 < ntiles) publish(t + 3, nk, nv, nb);
    lds_barrier();
    // buffer (t + 3) % 4 held tile t - 1, finished by every wave before this barrier
    if (t + 3 < ntiles) issue(t + 3);
    if (wave == 0 && t + 4 < ntiles) resolve(t + 4, nk, nv, nb);
    if (!wvalid) continue;  // uniform: a loader-only wave
    // a full tile of near-window keys past the first has all biases 0
    if (t > 0 && c0 + (t + 1) * AT_KEYS <= min(c1n, aa.n_near))
      compute_tile(s_kv[buf][0], s_kv[buf][1], tb, std::false_type{});
    else
      compute_tile(s_kv[buf][0], s_kv[buf][1], tb, std::true_type{});
  }

  // Pseudo-token tiles formed in LDS (aa.gen): row (k, s) of K is
  // bf16(c_k + concat_g C^K_g[z_{s,g}]) (c_k alone when the slot has no
  // residual), the values k_materialize writes; likewise V.  The inputs of a
  // tile (the bank rows' float32 sums, 1 KiB per slot, and decode records of
  // its <= PS_SLOTS slots) go by DMA into one of three 16 KiB staging buffers
  // three tiles ahead, with PS_INSTR load instructions per tile spread evenly
  // over the waves (unused ones repeat a valid slot), so every wave's
  // outstanding count is known; two tiles ahead the sums are turned into
  // centres in place.  Iteration t: wait for tile t+2's inputs, barrier,
  // issue tile t+3's, convert tile t+2's, form tile t+1 into buffer
  // (t+1) % 2, compute tile t: the forming of the next tile overlaps the
  // MFMA work of the current one.
  // LDS: buffers 0, 1 the formed tiles, s_kv[2][0] the unit's codebooks (16
  // KiB), s_kv[2][1] .. s_kv[3][1] the staging buffers.
  const int ps0 = min(aa.n_far, split * aa.far_chunk), ps1 = min(aa.n_far, ps0 + aa.far_chunk);
  const int npt = aa.gen && ps1 > ps0 ? (ps1 - ps0 + AT_KEYS - 1) / AT_KEYS : 0;
  if (npt > 0) {  // uniform
    constexpr int PS_INSTR = 16;                        // PS_SLOTS centre loads + 2 record loads
    constexpr int PS_STAGE = AT_TILE_BYTES;             // 16 KiB
    constexpr int PS_REC = PS_SLOTS * 1024;             // records at this offset of a stage
    constexpr int IPW = PS_INSTR / NW;                  // load instructions per wave per tile
    constexpr int CPT = 2 * AT_KEYS * 16 / (NW * 64);   // 16-byte chunks formed per thread per tile
    static_assert(PS_REC + 2 * 1024 <= PS_STAGE && 2 * PCW * 4 * PS_SLOTS <= 2 * 1024, "stage layout");
    static_assert(1024 % (NW * 64) == 0, "a thread's chunks of one pass are all K or all V");
    const int S = dm.S;
    const float invS2 = 1.0f / (float)S;
    auto divS = [&](int x) {
      int k = (int)((float)x * invS2);
      k -= k * S > x ? 1 : 0;
      k += (k + 1) * S <= x ? 1 : 0;
      return k;
    };
    uint8_t* s_cbb = s_kv[2][0];
    uint8_t* s_stage = s_kv[2][1];
    const size_t ubase = (size_t)u * dm.K;
    // Staged centre of the slot at stage position i: 16-byte unit (K/V half
    // kvh, part 2 cl + e) at kvh * 32 + (2 cl + e + 2 i) % 32, so that rows of
    // different slots reading one chunk fall on different banks.
    auto stage = [&](int t) {
      const int r0 = ps0 + t * AT_KEYS;
      const int kA = divS(r0), kB = divS(min(r0 + AT_KEYS, ps1) - 1);
      const int nk = kB - kA + 1;
      uint8_t* sb = s_stage + (t % 3) * PS_STAGE;
#pragma unroll
      for (int q = 0; q < IPW; ++q) {
        const int i = wave + q * NW;  // uniform
        const uint8_t* src;
        uint8_t* dst;
        if (i < PS_SLOTS) {
          const int part = (lane & 32) + (((lane & 31) - 2 * i) & 31);
          src = ws.bank + (unit * dm.K + kA + min(i, nk - 1)) * ROW + ROW_SUMK + part * 16;
          dst = sb + i * 1024;
        } else {
          const int ch = min((i - PS_SLOTS) * 64 + lane, nk * (2 * PCW / 4) - 1);
          src = reinterpret_cast<const uint8_t*>(ws.pcodes + (ubase + kA) * 2 * PCW) + ch * 16;
          dst = sb + PS_REC + (i - PS_SLOTS) * 1024;
        }
        lds_dma16(src, dst);
      }
    };
    // The staged sums of tile t's slots become their float32 centres
    // sum / n (IEEE division; EMA centres are stored as such) in place, n
    // from the staged value records.
    const bool ema = (dm.flags & PROTOKV_FLAG_EMA_CENTRES) != 0;
    auto convert = [&](int t) {
      const int r0 = ps0 + t * AT_KEYS;
      const int kA = divS(r0), kB = divS(min(r0 + AT_KEYS, ps1) - 1);
      const int nk = kB - kA + 1;
      uint8_t* sb = s_stage + (t % 3) * PS_STAGE;
      const uint32_t* recs = reinterpret_cast<const uint32_t*>(sb + PS_REC);
      for (int x = tid; x < nk * 64; x += NW * 64) {
        const int i = x >> 6;
        float4* c4 = reinterpret_cast<float4*>(sb + i * 1024) + (x & 63);
        const float nf = ema ? 1.f : (float)recs[(i * 2 + 1) * PCW + SMAX + 1];
        const float4 v = *c4;
        *c4 = make_float4(v.x / nf, v.y / nf, v.z / nf, v.w / nf);
      }
    };
    // Tile t from stage t % 3 into buffer t % 2, in the layouts of the near
    // tiles.  A thread forms the 16-byte store units q = tid + e * NW * 64 of
    // K (row q % 64, chunk q / 64) and of V (row q / 4 % 64, chunk
    // 4 (q / 256) + q % 4): one K row and one V row per thread, and each
    // store instruction writes 1 KiB contiguous.  The K chunks of a thread
    // come in rotate-half pairs (chunk c and c + 8 hold dims i and i + D/2),
    // so with rotary positions each formed key, rounded to bf16 as written,
    // is turned at tau_k in registers (float32, the roundings of
    // k_materialize16) and rounded again.
    const bool rope = ws.rope_inv != nullptr;  // uniform
    auto form = [&](int t) {
      constexpr int UPT = 1024 / (NW * 64);  // units per thread of K (and of V)
      const int r0 = ps0 + t * AT_KEYS;
      const int kA = divS(r0);
      const uint8_t* sb = s_stage + (t % 3) * PS_STAGE;
      const int pb = t & 1;
      // the 8 values c + m w of 16-byte unit q (chunk cl) of the row of slot
      // j, tuple tup, as float
      auto unit8 = [&](int kv, int q, int cl, int j, uint32_t tup, float m, const float4* cen, float (&x)[8]) {
        const float4 ca = cen[(2 * cl + 2 * j) & 31], cb = cen[(2 * cl + 1 + 2 * j) & 31];
        const int g = cl >> 1;
        const int z = (tup >> (4 * (G - 1 - g))) & 15;
        const float4* cw = reinterpret_cast<const float4*>(s_cbb) + ((kv * G + g) * CMAX + z) * 4;
        const int zr = z >> 2;
        const float4 wa = cw[(2 * (cl & 1) + zr) & 3], wb = cw[(2 * (cl & 1) + 1 + zr) & 3];
        // w * m + c is exactly c + w (m = 1) or c (m = 0)
        x[0] = fmaf(wa.x, m, ca.x); x[1] = fmaf(wa.y, m, ca.y); x[2] = fmaf(wa.z, m, ca.z); x[3] = fmaf(wa.w, m, ca.w);
        x[4] = fmaf(wb.x, m, cb.x); x[5] = fmaf(wb.y, m, cb.y); x[6] = fmaf(wb.z, m, cb.z); x[7] = fmaf(wb.w, m, cb.w);
      };
      auto store8 = [&](int kv, int q, const float (&x)[8]) {
        const bf16x2 o0 = {(__bf16)x[0], (__bf16)x[1]}, o1 = {(__bf16)x[2], (__bf16)x[3]};
        const bf16x2 o2 = {(__bf16)x[4], (__bf16)x[5]}, o3 = {(__bf16)x[6], (__bf16)x[7]};
        *reinterpret_cast<uint4*>(s_kv[pb][kv] + q * 16) =
            make_uint4(__builtin_bit_cast(uint32_t, o0), __builtin_bit_cast(uint32_t, o1),
                       __builtin_bit_cast(uint32_t, o2), __builtin_bit_cast(uint32_t, o3));
      };
#pragma unroll
      for (int kv = 0; kv < 2; ++kv) {
        const int row = kv ? (tid >> 2) & 63 : tid & 63;
        const bool valid = r0 + row < ps1;
        const int prow = valid ? r0 + row : r0;  // rows past the context repeat a valid row (bias -inf)
        const int k = divS(prow);
        const int j = k - kA, s2 = prow - k * S;
        const uint32_t* rec = reinterpret_cast<const uint32_t*>(sb + PS_REC) + (j * 2 + kv) * PCW;
        const uint32_t tup = rec[s2];
        const float m = rec[SMAX] != 0u ? 0.f : 1.f;  // no residual: the centre alone
        const float4* cen = reinterpret_cast<const float4*>(sb + j * 1024 + kv * 512);
        if (kv == 0 && rope) {
          // K units e and e + UPT/2: chunks cl < 8 and cl + 8
#pragma unroll
          for (int e = 0; e < UPT / 2; ++e) {
            const int ql = tid + e * NW * 64, qh = ql + (UPT / 2) * NW * 64;
            const int cl = ql >> 6;
            float xl[8], xh[8];
            unit8(0, ql, cl, j, tup, m, cen, xl);
            unit8(0, qh, cl + 8, j, tup, m, cen, xh);
            const float4* cs = reinterpret_cast<const float4*>(&s_rtab[pb][j][8 * cl]);
#pragma unroll
            for (int i2 = 0; i2 < 4; ++i2) {
              const float4 a = cs[i2];  // (cos, sin) of pair indices 8 cl + 2 i2, + 1
#pragma unroll
              for (int h = 0; h < 2; ++h) {
                const int i = 2 * i2 + h;
                const float c = h ? a.z : a.x, sn = h ? a.w : a.y;
                const float x1 = (float)(__bf16)xl[i], x2 = (float)(__bf16)xh[i];
                float lo, hi;
                rope_pair(x1, x2, c, sn, lo, hi);
                xl[i] = lo;
                xh[i] = hi;
              }
            }
            store8(0, ql, xl);
            store8(0, qh, xh);
          }
        } else {
#pragma unroll
          for (int e = 0; e < UPT; ++e) {
            const int q = tid + e * NW * 64;
            const int cl = kv ? (q >> 8) * 4 + (q & 3) : q >> 6;
            float x[8];
            unit8(kv, q, cl, j, tup, m, cen, x);
            store8(kv, q, x);
          }
        }
        if (kv == 0 && tid < AT_KEYS)  // row == tid
          s_bias[pb][row] = valid ? (pb_lds ? s_pb[k] : ws.pbias[ubase + k] * LOG2E) : -INFINITY;
      }
    };
    // (cos, sin) table of tile t's slots from tau_k in the staged key
    // records (stage t % 3), into table t % 2: a thread's pair index i =
    // tid % 64 is the same for every entry it computes
    const double rinv = rope ? ws.rope_inv[tid & 63] : 0.0;
    auto rtab = [&](int t) {
      const int r0 = ps0 + t * AT_KEYS;
      const int kA = divS(r0), kB = divS(min(r0 + AT_KEYS, ps1) - 1);
      const int nk = kB - kA + 1;
      const uint32_t* recs = reinterpret_cast<const uint32_t*>(s_stage + (t % 3) * PS_STAGE + PS_REC);
      for (int x = tid; x < nk * 64; x += NW * 64) {
        const int jj = x >> 6;
        const double tau = (double)(int32_t)recs[jj * 2 * PCW + SMAX + 1];
        float c, sn;
        rope_cs(tau, rinv, c, sn);
        s_rtab[t & 1][jj][tid & 63] = make_float2(c, sn);
      }
    };

    lds_barrier();  // every wave is done with the near tiles (buffers and bias entries are reused)
    // codebooks as [K/V][subspace][codeword][4 parts of 16 bytes], part s of
    // codeword z at position (s + z / 4) % 4: rows reading one chunk of
    // different codewords fall on different banks
#pragma unroll
    for (int q = 0; q < 16 / NW; ++q) {
      const int i = wave + q * NW;
      const int pos = i * 64 + lane;
      const int z = (pos >> 2) & 15;
      const int part = (pos & ~3) + (((pos & 3) - (z >> 2)) & 3);
      lds_dma16(reinterpret_cast<const uint8_t*>(ws.codebooks + unit * (2 * G * CMAX * DP)) + part * 16,
                s_cbb + i * 1024);
    }
    stage(0);
    if (npt > 1) stage(1);
    if (npt > 2) stage(2);
    // codebooks and tiles 0 and 1's inputs have landed (tile 2's may be in
    // flight): both are converted (and with rotary positions get their
    // tables) before tile 0 is formed
    if (npt > 2) wait_vm<IPW>();
    else wait_vm<0>();
    lds_barrier();
    convert(0);
    if (npt > 1) convert(1);
    if (rope) {
      rtab(0);
      if (npt > 1) rtab(1);
    }
    lds_barrier();
    form(0);
    for (int t = 0; t < npt; ++t) {
      // this wave's loads of tile t+2's inputs have landed (converted, and
      // with rotary positions tabled, now; tile t+1's were converted in the
      // previous iteration)
      wait_vm<0>();
      // tile t formed everywhere; stage t % 3 (read by form(t)), formed
      // buffer (t+1) % 2 (read by compute(t-1)) and table t % 2 (read by
      // form(t)) are free
      lds_barrier();
      if (t + 3 < npt) stage(t + 3);
      if (t + 2 < npt) convert(t + 2);
      if (rope && t + 2 < npt) rtab(t + 2);
      // waves w and w + 4 share a SIMD: one forms before computing, the other
      // after, so the forming overlaps the partner's matrix work
      const bool form_first = wave < 4 || !wvalid;  // uniform
      if (form_first && t + 1 < npt) form(t + 1);
      if (wvalid) compute_tile(s_kv[t & 1][0], s_kv[t & 1][1], t & 1, std::true_type{});
      if (!form_first && t + 1 < npt) form(t + 1);
    }
  }
  if constexpr (KH == 2) {
    // waves of key half 1 hand (reference, sum, O) to their half-0 partner
    // through LDS; both are relative to their own reference, so
    // O = 2^(m1 - m) O1 + 2^(m2 - m) O2, l likewise, m = max(m1, m2)
    __syncthreads();  // every wave is done with the tiles (LDS reused)
    float* s_part = reinterpret_cast<float*>(&s_kv[0][0][0]) + (size_t)rblk * 66 * 64;
    if (kh == 1) {
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) s_part[(b * 16 + i) * 64 + lane] = oacc[b][i];
      s_part[64 * 64 + lane] = mref;
      s_part[65 * 64 + lane] = lrun;
    }
    __syncthreads();
    if (kh == 1) return;
    const float m2 = s_part[64 * 64 + lane], l2 = s_part[65 * 64 + lane];
    const float m = fmaxf(mref, m2);
    const float a1 = __builtin_amdgcn_exp2f(mref - m), a2 = __builtin_amdgcn_exp2f(m2 - m);
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[b][i] = oacc[b][i] * a1 + s_part[(b * 16 + i) * 64 + lane] * a2;
    lrun = lrun * a1 + l2 * a2;
    mref = m;
  }
  const float mrun = mref;

  const size_t orow_t = rvalid ? (size_t)(r / grp) : 0;
  const int ogg = rvalid ? r % grp : 0;
  const size_t orow = (((size_t)l * aa.tq + orow_t) * dm.Hq + kvh * grp + ogg) * D;
  if (aa.splits == 1) {
    if (rvalid) {
      const float inv = lrun > 0.f ? 1.0f / lrun : 0.f;
      uint16_t* o = reinterpret_cast<uint16_t*>(aa.o) + orow;
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[b * 32 + (i >> 2) * 8 + half * 4 + (i & 3)] = q_to_bf16(oacc[b][i] * inv);
      if (half == 0 && aa.lse) aa.lse[((size_t)l * aa.tq + orow_t) * dm.Hq + kvh * grp + ogg] = (mrun + log2f(lrun)) * LN2;
    }
    return;
  }
  if (rvalid) {
    float* po = ws.part_o + (((size_t)u * dm.max_splits + split) * dm.max_rows + r) * D;
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) po[b * 32 + (i >> 2) * 8 + half * 4 + (i & 3)] = oacc[b][i];
    if (half == 0) {
      float* pml = ws.part_ml + (((size_t)u * dm.max_splits + split) * dm.max_rows + r) * 2;
      pml[0] = mrun;
      pml[1] = lrun;
    }
  }
}

// Combines the splits of each query row: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
// Combines the splits' partials of output row r, dims 4 d4 .. 4 d4 + 3, of
// kv head u: O = sum_s w_s O_s / sum_s w_s l_s with w_s = 2^(m_s - max m).
// NSP: the number of splits when known at compile time (0: aa.splits).
template <int FP32, int NSP>
__device__ __forceinline__ void merge_row4(const Dims& dm, const Workspace& ws, const AttendArgs& aa, int u, int r,
                                           int d4) {
  constexpr int NS = NSP ? NSP : MAX_SPLITS;
  const int nsplit = NSP ? NSP : aa.splits;
  const int grp = dm.Hq / dm.Hkv;
  const int l = u / dm.Hkv, kvh = u % dm.Hkv;
  float ms[NS], ls[NS];
  float4 ov[NS];
  float M = -INFINITY;
#pragma unroll
  for (int s2 = 0; s2 < NS; ++s2) {
    if (s2 < nsplit) {
      const size_t pr = ((size_t)u * dm.max_splits + s2) * dm.max_rows + r;
      ms[s2] = ws.part_ml[pr * 2];
      ls[s2] = ws.part_ml[pr * 2 + 1];
      ov[s2] = reinterpret_cast<const float4*>(ws.part_o + pr * D)[d4];
      M = fmaxf(M, ms[s2]);
    }
  }
  float Lsum = 0.f;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int s2 = 0; s2 < NS; ++s2) {
    if (s2 < nsplit) {
      const float w = ms[s2] == -INFINITY ? 0.f : exp2f(ms[s2] - M);
      Lsum += w * ls[s2];
      o.x += w * ov[s2].x;
      o.y += w * ov[s2].y;
      o.z += w * ov[s2].z;
      o.w += w * ov[s2].w;
    }
  }
  const float inv = Lsum > 0.f ? 1.0f / Lsum : 0.f;
  const int t = r / grp, gg = r % grp;
  const size_t orow = (((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg) * D;
  if (FP32) {
    reinterpret_cast<float4*>(reinterpret_cast<float*>(aa.o) + orow)[d4] =
        make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
  } else {
    const uint2 packed = make_uint2((uint32_t)q_to_bf16(o.x * inv) | ((uint32_t)q_to_bf16(o.y * inv) << 16),
                                    (uint32_t)q_to_bf16(o.z * inv) | ((uint32_t)q_to_bf16(o.w * inv) << 16));
    reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(aa.o) + orow)[d4] = packed;
  }
  if (d4 == 0 && aa.lse) aa.lse[((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg] = (M + log2f(Lsum)) * LN2;
}

template <int FP32, int NSP>
__global__ __launch_bounds__(256) void k_attend_merge(Dims dm, Workspace ws, AttendArgs aa, int rows) {
  // thread = (kv head, query row, 4 output dims); every split's (m, l) and
  // partial O are loaded together (units * rows * D / 4 < 2^31)
  const int gt = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (gt >= dm.units * rows * (D / 4)) return;
  const int d4 = gt & (D / 4 - 1);
  const int rr = gt / (D / 4);
  const int r = rr % rows;
  const int u = rr / rows;
  merge_row4<FP32, NSP>(dm, ws, aa, u, r, d4);
}

// float32 path (small fp32 streams): one wave per (kv head, query row, split),
// each context key scored by the whole wave (two components per lane).
__global__ __launch_bounds__(64) void k_attend_f32(Dims dm, Workspace ws, AttendArgs aa, int rows) {
  const int lane = threadIdx.x;
  const int split = blockIdx.x % aa.splits;
  const int r = (blockIdx.x / aa.splits) % rows;
  const int u = blockIdx.x / (aa.splits * rows);
  const size_t unit = (size_t)aa.sid * dm.units + u;
  const int grp = dm.Hq / dm.Hkv;
  const int l = u / dm.Hkv, kvh = u % dm.Hkv;
  const int t = r / grp, gg = r % grp;
  const float2 qv = reinterpret_cast<const float2*>(reinterpret_cast<const float*>(aa.q) +
                                                    (((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg) * D)[lane];
  const int ctx = aa.n_near + aa.n_far;
  const int c0 = split * aa.chunk, c1 = min(ctx, c0 + aa.chunk);
  const float scale = LOG2E / sqrtf((float)D);
  float mrun = -INFINITY, lrun = 0.f, o0 = 0.f, o1 = 0.f;
  for (int idx = c0; idx < c1; ++idx) {
    CtxRef kr = ctx_key<4>(dm, ws, aa, unit, u, idx, false);
    CtxRef vr = ctx_key<4>(dm, ws, aa, unit, u, idx, true);
    const float2 kv = reinterpret_cast<const float2*>(kr.base)[lane];
    float dot = qv.x * kv.x + qv.y * kv.y;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) dot += __shfl_xor(dot, o, 64);
    const float s = dot * scale + kr.bias * LOG2E;
    const float mnew = fmaxf(mrun, s);
    const float alpha = exp2f(mrun - mnew);
    const float p = exp2f(s - mnew);
    const float2 vv = reinterpret_cast<const float2*>(vr.base)[lane];
    lrun = lrun * alpha + p;
    o0 = o0 * alpha + p * vv.x;
    o1 = o1 * alpha + p * vv.y;
    mrun = mnew;
  }
  const size_t pr = ((size_t)u * dm.max_splits + split) * dm.max_rows + r;
  reinterpret_cast<float2*>(ws.part_o + pr * D)[lane] = make_float2(o0, o1);
  if (lane == 0) {
    ws.part_ml[pr * 2] = mrun;
    ws.part_ml[pr * 2 + 1] = lrun;
  }
}

hipError_t launch_attend(const Dims& dm, const Workspace& ws, const AttendArgs& aa, hipStream_t st) {
  const int grp = dm.Hq / dm.Hkv;
  const int rows = aa.tq * grp;
  if (dm.kv_fp32) {
    hipLaunchKernelGGL(k_attend_f32, dim3(dm.units * rows * aa.splits), dim3(64), 0, st, dm, ws, aa, rows);
  } else {
    // 8 waves per workgroup: 256 query rows, or at most 128 rows with the
    // tiles' key halves split between wave pairs
    const int rblocks = (rows + AT_ROWS - 1) / AT_ROWS;
    if (rows > 128)
      hipLaunchKernelGGL((k_attend_bf16<8, 1>), dim3(dm.units * aa.splits * rblocks), dim3(512), 0, st, dm, ws, aa,
                         rows, rblocks);
    else
      hipLaunchKernelGGL((k_attend_bf16<8, 2>), dim3(dm.units * aa.splits), dim3(512), 0, st, dm, ws, aa, rows, 1);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scratch of protokv_attend_static (callers that cannot allocate): the split
// partials and the rotated query live in this file-scope device array instead
// of the workspace.  Every device the library runs on holds its own copy
// until the process ends; host code must use the address from
// static_scratch_ptr, never the array's name.
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[PROTOKV_STATIC_SCRATCH_BYTES];

hipError_t static_scratch_ptr(void** out) {
  static std::mutex mu;
  static void* per_device[MAX_DEVICES] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!per_device[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    per_device[dev] = p;
  }
  *out = per_device[dev];
  return hipSuccess;
}

hipError_t launch_attend_merge(const Dims& dm, const Workspace& ws, const AttendArgs& aa, hipStream_t st) {
  if (!dm.kv_fp32 && aa.splits == 1) return hipSuccess;  // the bf16 readout wrote O directly
  const int rows = aa.tq * (dm.Hq / dm.Hkv);
  const int nb = (int)(((size_t)dm.units * rows * (D / 4) + 255) / 256);
  if (dm.kv_fp32)
    hipLaunchKernelGGL((k_attend_merge<1, 0>), dim3(nb), dim3(256), 0, st, dm, ws, aa, rows);
  else if (aa.splits == 2)
    hipLaunchKernelGGL((k_attend_merge<0, 2>), dim3(nb), dim3(256), 0, st, dm, ws, aa, rows);
  else
    hipLaunchKernelGGL((k_attend_merge<0, 0>), dim3(nb), dim3(256), 0, st, dm, ws, aa, rows);
  return hipGetLastError();
}

}  // namespace pkv
