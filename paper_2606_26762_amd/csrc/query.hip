// Query path of libprotokv for gfx950: pseudo-token synthesis and the
// mass-aware readout.
//
// Paper: Section "Residual Statistics and Pseudo-Token Interface" (pseudo
// tokens, mass-aware bias, Eq. attn_logit), Eq. pq and Appendix Algorithms
// "DecodeTopSResidualModes" and "ProtoKV Query-Time Pseudo-Token Decoding
// and Attention".
#include "pkv_internal.h"

namespace pkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t q_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float q_from_bf16(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

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

// One wave per workgroup over 32 prototypes of one (layer, kv head): lanes
// 0-31 decode the key histograms, lanes 32-63 the value histograms, then the
// wave writes the pseudo-tokens row by row (lane l writes components 2l, 2l+1).
template <int FP32>
__global__ __launch_bounds__(64) void k_synthesize(Dims dm, Workspace ws, int sid, int n_active,
                                                   int blocks_per_unit) {
  extern __shared__ __attribute__((aligned(16))) uint8_t s_dyn[];
  __shared__ uint32_t s_codes[2][SYN_P][SMAX];
  __shared__ uint32_t s_nores[2][SYN_P];  // 1: no residual statistics, S copies of the centre
  const int lane = threadIdx.x;
  const int u = blockIdx.x / blocks_per_unit;
  const int p0 = (blockIdx.x % blocks_per_unit) * SYN_P;
  const size_t unit = (size_t)sid * dm.units + u;
  const int S = dm.S;
  const bool pq = (dm.flags & PROTOKV_FLAG_PQ) != 0;
  BeamView bv;
  bv.S = S;
  bv.w0 = reinterpret_cast<uint64_t*>(s_dyn);
  bv.w1 = bv.w0 + 2 * S * 64;
  bv.w2 = bv.w1 + 2 * S * 64;
  bv.code = reinterpret_cast<uint32_t*>(bv.w2 + 2 * S * 64);
  const float* cbk = ws.codebooks + unit * (2 * G * CMAX * DP);

  const int pl = lane & 31, kv = lane >> 5;
  const int p = p0 + pl;
  if (p < n_active) {
    const uint8_t* row = ws.bank + (unit * dm.K + p) * ROW;
    const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
    if (pq && m.n_res > 0) {
      const uint32_t* hist = reinterpret_cast<const uint32_t*>(row + (kv ? ROW_HV : ROW_HK));
      uint32_t codes[SMAX];
      decode_top_s(hist, dm.C, S, bv, lane, codes);
      for (int s = 0; s < S; ++s) s_codes[kv][pl][s] = codes[s];
      s_nores[kv][pl] = 0u;
    } else {
      s_nores[kv][pl] = 1u;
    }
    if (kv == 0) {
      const bool mb = (dm.flags & PROTOKV_FLAG_MASS_BIAS) != 0;
      ws.pbias[(size_t)u * dm.K + p] = mb ? logf((float)m.n) : 0.f;
    }
  }
  __syncthreads();

  const size_t es = FP32 ? 4 : 2;
  const int g = lane >> 3, u16 = (2 * lane) & 15;
  for (int q = 0; q < SYN_P; ++q) {
    const int pp = p0 + q;
    if (pp >= n_active) break;
    const uint8_t* row = ws.bank + (unit * dm.K + pp) * ROW;
    const RowMeta m = *reinterpret_cast<const RowMeta*>(row + ROW_META);
    const float nf = (float)m.n;
    const float2 sk = reinterpret_cast<const float2*>(row + ROW_SUMK)[lane];
    const float2 sv = reinterpret_cast<const float2*>(row + ROW_SUMV)[lane];
    const float2 ck = make_float2(sk.x / nf, sk.y / nf);
    const float2 cv = make_float2(sv.x / nf, sv.y / nf);
    for (int w = 0; w < 2; ++w) {
      const float2 c = w ? cv : ck;
      uint8_t* out = (w ? ws.pv : ws.pk) + ((size_t)u * dm.K * S + (size_t)pp * S) * D * es;
      const bool nores = s_nores[w][q] != 0u;
      for (int s = 0; s < S; ++s) {
        const uint32_t code = s_codes[w][q][s];
        float2 val = c;
        if (!nores) {
          const int z = (code >> (4 * (G - 1 - g))) & 15;
          const float2 cw = *reinterpret_cast<const float2*>(cbk + ((w * G + g) * CMAX + z) * DP + u16);
          val.x = c.x + cw.x;
          val.y = c.y + cw.y;
        }
        if (FP32) {
          reinterpret_cast<float2*>(out + (size_t)s * D * 4)[lane] = val;
        } else {
          const uint32_t packed = (uint32_t)q_to_bf16(val.x) | ((uint32_t)q_to_bf16(val.y) << 16);
          reinterpret_cast<uint32_t*>(out + (size_t)s * D * 2)[lane] = packed;
        }
      }
    }
  }
}

hipError_t launch_synthesize(const Dims& dm, const Workspace& ws, int sid, int n_active, hipStream_t st) {
  if (n_active <= 0) return hipSuccess;
  int bpu = (n_active + SYN_P - 1) / SYN_P;
  dim3 grid(dm.units * bpu);
  size_t lds = (size_t)2 * dm.S * 64 * (3 * sizeof(uint64_t) + sizeof(uint32_t));
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_synthesize<1>, grid, dim3(64), lds, st, dm, ws, sid, n_active, bpu);
  else
    hipLaunchKernelGGL(k_synthesize<0>, grid, dim3(64), lds, st, dm, ws, sid, n_active, bpu);
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
constexpr int KROW = 136;  // staged key row (bf16), 128 + 8 padding
constexpr int VCOL = 40;   // staged transposed value row (bf16), 32 keys + 8 padding

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
    r.base = (values ? ws.ring_v : ws.ring_k) + (((unit * (dm.W + 1) + slot) * dm.T + tok) * (size_t)D) * ES;
  } else {
    const int row = idx - aa.n_near;
    r.base = (values ? ws.pv : ws.pk) + (((size_t)u * dm.K * dm.S + row) * (size_t)D) * ES;
    r.bias = ws.pbias[(size_t)u * dm.K + row / dm.S];
  }
  return r;
}

// bf16 path: workgroup = one (kv head, context split), one wave per 32 query
// rows.  S^T = K Q^T and O^T = V^T P with v_mfma_f32_32x32x16_bf16; each lane
// holds one query column, so the online softmax needs only lane-local work
// plus one exchange with the partner lane (the other 16 key rows).
__global__ __launch_bounds__(1024) void k_attend_bf16(Dims dm, Workspace ws, AttendArgs aa, int rows) {
  __shared__ __attribute__((aligned(16))) uint16_t s_k[2][32 * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t s_vt[2][D * VCOL];
  __shared__ float s_bias[2][32];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nthr = blockDim.x;
  const int split = blockIdx.x % aa.splits;
  const int u = blockIdx.x / aa.splits;
  const size_t unit = (size_t)aa.sid * dm.units + u;
  const int grp = dm.Hq / dm.Hkv;
  const int l = u / dm.Hkv, kvh = u % dm.Hkv;
  const int ctx = aa.n_near + aa.n_far;
  const int c0 = split * aa.chunk;
  const int c1 = min(ctx, c0 + aa.chunk);
  const int ntiles = c1 > c0 ? (c1 - c0 + 31) / 32 : 0;

  const int col = lane & 31, half = lane >> 5;
  const int r = wave * 32 + col;  // query row of this lane
  const bool rvalid = r < rows;
  // Q^T operand: dims kk*16 + half*8 + 0..7 of row r.
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
  const float scale = LOG2E / sqrtf((float)D);
  f32x16 oacc[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) oacc[b] = (f32x16){0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;

  auto stage = [&](int t, int buf) {
    const int base = c0 + t * 32;
    // keys: 32 rows x 16 chunks of 16 B
    for (int c = tid; c < 32 * 16; c += nthr) {
      const int rr = c >> 4, cc = c & 15;
      const int idx = base + rr;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (idx < c1) {
        CtxRef kr = ctx_key<2>(dm, ws, aa, unit, u, idx, false);
        val = *reinterpret_cast<const uint4*>(kr.base + cc * 16);
      }
      *reinterpret_cast<uint4*>(s_k[buf] + rr * KROW + cc * 8) = val;
    }
    // values, transposed into [dim][key]
    for (int c = tid; c < 32 * 16; c += nthr) {
      const int rr = c >> 4, cc = c & 15;
      const int idx = base + rr;
      u16x8 val = (u16x8)0;
      if (idx < c1) {
        CtxRef vr = ctx_key<2>(dm, ws, aa, unit, u, idx, true);
        val = *reinterpret_cast<const u16x8*>(vr.base + cc * 16);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) s_vt[buf][(cc * 8 + i) * VCOL + rr] = val[i];
    }
    if (tid < 32) {
      const int idx = base + tid;
      float bval = -INFINITY;
      if (idx < c1) bval = ctx_key<2>(dm, ws, aa, unit, u, idx, false).bias;
      s_bias[buf][tid] = bval;
    }
  };

  if (ntiles > 0) stage(0, 0);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) stage(t + 1, buf ^ 1);
    // S^T = K Q^T: rows = keys (m), columns = query rows
    f32x16 sacc = (f32x16){0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t* kr = s_k[buf] + col * KROW + half * 8;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const bf16x8 ak = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(kr + kk * 16));
      sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak, bq[kk], sacc, 0, 0, 0);
    }
    // logits in log2 units, masked beyond the context
    float tmax = -INFINITY;
    float sv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int m = (i >> 2) * 8 + half * 4 + (i & 3);
      const float bsv = s_bias[buf][m];
      const float x = bsv == -INFINITY ? -INFINITY : sacc[i] * scale + bsv * LOG2E;
      sv[i] = x;
      tmax = fmaxf(tmax, x);
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(mrun, tmax);
    const float alpha = mnew == -INFINITY ? 1.f : exp2f(mrun - mnew);
    float psum = 0.f;
    u16x8 pb0, pb1;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float pv = sv[i] == -INFINITY ? 0.f : exp2f(sv[i] - mnew);
      psum += pv;
      const uint16_t hb = q_to_bf16(pv);
      if (i < 8) pb0[i] = hb; else pb1[i - 8] = hb;
    }
    psum += __shfl_xor(psum, 32, 64);
    lrun = lrun * alpha + psum;
    mrun = mnew;
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[b][i] *= alpha;
    const bf16x8 bp0 = __builtin_bit_cast(bf16x8, pb0), bp1 = __builtin_bit_cast(bf16x8, pb1);
    // O^T = V^T P: A = V^T rows (dims), k positions half*8 + i <-> keys
    // {4 half + 0..3, 8 + 4 half + 0..3} (+16 for the second step).
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const uint16_t* vr = s_vt[buf] + (b * 32 + col) * VCOL + 4 * half;
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const u16x4 lo = *reinterpret_cast<const u16x4*>(vr + st * 16);
        const u16x4 hi = *reinterpret_cast<const u16x4*>(vr + st * 16 + 8);
        const u16x8 a = (u16x8){lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        oacc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                          st ? bp1 : bp0, oacc[b], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // partial (unnormalised O, running max in log2 units, sum)
  if (rvalid) {
    float* po = ws.part_o + (((size_t)u * dm.max_splits + split) * dm.max_rows + r) * D;
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int dim = b * 32 + (i >> 2) * 8 + half * 4 + (i & 3);
        po[dim] = oacc[b][i];
      }
    if (half == 0) {
      float* pml = ws.part_ml + (((size_t)u * dm.max_splits + split) * dm.max_rows + r) * 2;
      pml[0] = mrun;
      pml[1] = lrun;
    }
  }
}

// Combines the splits of each query row: O = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
template <int FP32>
__global__ __launch_bounds__(64) void k_attend_merge(Dims dm, Workspace ws, AttendArgs aa, int rows) {
  const int lane = threadIdx.x;
  const int r = blockIdx.x % rows;
  const int u = blockIdx.x / rows;
  const int grp = dm.Hq / dm.Hkv;
  const int l = u / dm.Hkv, kvh = u % dm.Hkv;
  float M = -INFINITY;
  for (int s = 0; s < aa.splits; ++s)
    M = fmaxf(M, ws.part_ml[(((size_t)u * dm.max_splits + s) * dm.max_rows + r) * 2]);
  float Lsum = 0.f, o0 = 0.f, o1 = 0.f;
  for (int s = 0; s < aa.splits; ++s) {
    const size_t pr = ((size_t)u * dm.max_splits + s) * dm.max_rows + r;
    const float ms = ws.part_ml[pr * 2], ls = ws.part_ml[pr * 2 + 1];
    const float w = ms == -INFINITY ? 0.f : exp2f(ms - M);
    Lsum += w * ls;
    const float2 ov = reinterpret_cast<const float2*>(ws.part_o + pr * D)[lane];
    o0 += w * ov.x;
    o1 += w * ov.y;
  }
  const float inv = Lsum > 0.f ? 1.0f / Lsum : 0.f;
  const int t = r / grp, gg = r % grp;
  const size_t orow = (((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg) * D;
  if (FP32) {
    reinterpret_cast<float2*>(reinterpret_cast<float*>(aa.o) + orow)[lane] = make_float2(o0 * inv, o1 * inv);
  } else {
    reinterpret_cast<uint32_t*>(reinterpret_cast<uint16_t*>(aa.o) + orow)[lane] =
        (uint32_t)q_to_bf16(o0 * inv) | ((uint32_t)q_to_bf16(o1 * inv) << 16);
  }
  if (lane == 0 && aa.lse) aa.lse[((size_t)l * aa.tq + t) * dm.Hq + kvh * grp + gg] = (M + log2f(Lsum)) * LN2;
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
    const int waves = (rows + 31) / 32;
    hipLaunchKernelGGL(k_attend_bf16, dim3(dm.units * aa.splits), dim3(waves * 64), 0, st, dm, ws, aa, rows);
  }
  return hipGetLastError();
}

hipError_t launch_attend_merge(const Dims& dm, const Workspace& ws, const AttendArgs& aa, hipStream_t st) {
  const int rows = aa.tq * (dm.Hq / dm.Hkv);
  if (dm.kv_fp32)
    hipLaunchKernelGGL(k_attend_merge<1>, dim3(dm.units * rows), dim3(64), 0, st, dm, ws, aa, rows);
  else
    hipLaunchKernelGGL(k_attend_merge<0>, dim3(dm.units * rows), dim3(64), 0, st, dm, ws, aa, rows);
  return hipGetLastError();
}

}  // namespace pkv
