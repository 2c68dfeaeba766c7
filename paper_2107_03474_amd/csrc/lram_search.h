// lram_search.h -- part of liblram (included by lram.hip only).
//
// The neighbour search (Sec. 2.6): phase A (wrap, closest point of Lambda, the
// signed permutation into F) and phase B (per-query tables, candidate scan,
// selection of the closest k, locations and weights).

#pragma once

namespace {

// ---------------------------------------------------------------------------
// Phase A: closest point of Lambda and the reduction into F (Sec. 2.6).

// Nearest point of D8 = {r in Z^8 : sum r even} to y: round every coordinate,
// and if the sum is odd re-round the coordinate that was worst rounded.
__device__ __forceinline__ void d8_round(const float (&y)[8], int (&r)[8]) {
  float dmax = -1.0f;
  int jmax = 0, s = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float ri = rintf(y[i]);
    r[i] = (int)ri;
    float d = fabsf(y[i] - ri);
    if (d > dmax) {
      dmax = d;
      jmax = i;
    }
    s += r[i];
  }
  if (s & 1) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i == jmax) r[i] += (y[i] > (float)r[i]) ? 1 : -1;
  }
}

// Input float4s per lookup: q (8 floats) or z (16, the activation layer).
template <bool TH>
constexpr int in_vec4() { return TH ? 4 : 2; }

// The query of one lookup and its output scale, from the lookup's input
// vectors v.  TH = false: q itself (8 floats), scale 1.  TH = true, the
// activation layer of Sec. 2.3: z_i = in[2i] + i in[2i+1], q_i = (K_i / 2 pi)
// arg z_i formed in fp64 and rounded once to fp32, scale (sum_i 1/|z_i|)^-1 (0
// when some z_i = 0); a non-finite input gives a NaN query (empty neighbour
// list) and scale 0.
template <bool TH>
__device__ __forceinline__ void query_from(const float4 (&v)[in_vec4<TH>()], const Params P, float (&qq)[8],
                                           float& scale) {
  if constexpr (!TH) {
    qq[0] = v[0].x; qq[1] = v[0].y; qq[2] = v[0].z; qq[3] = v[0].w;
    qq[4] = v[1].x; qq[5] = v[1].y; qq[6] = v[1].z; qq[7] = v[1].w;
    scale = 1.0f;
  } else {
    float z[16];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      z[4 * k] = v[k].x; z[4 * k + 1] = v[k].y; z[4 * k + 2] = v[k].z; z[4 * k + 3] = v[k].w;
    }
    bool finite = true;
    double inv = 0.0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const double a = z[2 * i], b = z[2 * i + 1];
      finite = finite && isfinite(z[2 * i]) && isfinite(z[2 * i + 1]);
      inv += 1.0 / sqrt(a * a + b * b);
      qq[i] = (float)(atan2(b, a) * P.cK[i]);
    }
    if (!finite) qq[0] = __builtin_nanf("");
    scale = finite ? (float)(1.0 / inv) : 0.0f;
  }
}

template <bool TH>
__device__ __forceinline__ void load_input(const float* __restrict__ in, float4 (&v)[in_vec4<TH>()]) {
#pragma unroll
  for (int k = 0; k < in_vec4<TH>(); ++k) v[k] = reinterpret_cast<const float4*>(in)[k];
}

template <bool TH>
__device__ __forceinline__ void load_query(const float* __restrict__ in, const Params P, float (&qq)[8],
                                           float& scale) {
  float4 v[in_vec4<TH>()];
  load_input<TH>(in, v);
  query_from<TH>(v, P, qq, scale);
}

// Wrapped Lambda-scale query x and the closest point c of Lambda (either coset);
// false for a non-finite query (x = 0 then).
__device__ __forceinline__ bool closest_point(const float (&qq)[8], bool have, const Params P, float (&x)[8],
                                              int (&c)[8]) {
  bool valid = have;
  if (have) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float xi = 2.0f * qq[i];
      if (!(xi >= 0.0f && xi < P.twoK[i])) xi = fmodf(xi, P.twoK[i]);
      valid = valid && isfinite(xi);
      x[i] = xi;
    }
  }
  if (!valid) {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = 0.0f;
  }
  // Lambda = 2 D8  u  (2 D8 + 1): decode both cosets at half scale.
  float y0[8], y1[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    y0[i] = x[i] * 0.5f;
    y1[i] = (x[i] - 1.0f) * 0.5f;
  }
  int r0[8], r1[8];
  d8_round(y0, r0);
  d8_round(y1, r1);
  float d0 = 0.0f, d1 = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float e0 = x[i] - (float)(2 * r0[i]);
    float e1 = x[i] - (float)(2 * r1[i] + 1);
    d0 += e0 * e0;
    d1 += e1 * e1;
  }
  const bool odd = d1 < d0;
#pragma unroll
  for (int i = 0; i < 8; ++i) c[i] = odd ? 2 * r1[i] + 1 : 2 * r0[i];
  return valid;
}

template <bool TH>
__device__ __forceinline__ void make_frame(const float* __restrict__ in, bool have, const Params P, Frame& F) {
  float x[8];
  int c[8];
  float qq[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float scale = 0.0f;
  if (have) load_query<TH>(in, P, qq, scale);
  const bool valid = closest_point(qq, have, P, x, c);
  float a[8];
  uint32_t neg = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float y = x[i] - (float)c[i];
    a[i] = fabsf(y);
    neg |= (y < 0.0f ? 1u : 0u) << i;
  }
  // rank of |y_i| in descending order (ties by index): F position of coordinate i
  uint32_t sel[8];
  int last = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int ri = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j != i) ri += (a[j] > a[i] || (a[j] == a[i] && j < i)) ? 1 : 0;
    sel[i] = 0x0C0C0C00u | (uint32_t)ri;
    if (ri == 7) last = i;
  }
  // only even numbers of sign changes are isometries of Lambda: fix the parity
  // on the coordinate that lands last (smallest |y|)
  if (__popc(neg) & 1) neg ^= 1u << last;
  float4* fx = reinterpret_cast<float4*>(F.x);
  fx[0] = make_float4(x[0], x[1], x[2], x[3]);
  fx[1] = make_float4(x[4], x[5], x[6], x[7]);
  uint4* fs = reinterpret_cast<uint4*>(F.sel);
  fs[0] = make_uint4(sel[0], sel[1], sel[2], sel[3]);
  fs[1] = make_uint4(sel[4], sel[5], sel[6], sel[7]);
  uint4 w;
  w.x = (uint32_t)(uint16_t)c[0] | ((uint32_t)(uint16_t)c[1] << 16);
  w.y = (uint32_t)(uint16_t)c[2] | ((uint32_t)(uint16_t)c[3] << 16);
  w.z = (uint32_t)(uint16_t)c[4] | ((uint32_t)(uint16_t)c[5] << 16);
  w.w = (uint32_t)(uint16_t)c[6] | ((uint32_t)(uint16_t)c[7] << 16);
  reinterpret_cast<uint4*>(F.c)[0] = w;
  reinterpret_cast<uint4*>(&F.misc)[0] = make_uint4(neg | (valid ? 0x100u : 0u), __float_as_uint(scale), 0u, 0u);
}

// ---------------------------------------------------------------------------
// Phase B: the neighbour search of one lookup.

// Packed candidate bytes: byte j = 4*(p_j - CMIN) + 64*w (the LDS byte offset of
// table entry (., w, p_j) within a coordinate's 256-byte block).
template <int LIST>
__device__ __forceinline__ bool load_candidate(int idx, uint32_t wbyte, uint32_t& lo, uint32_t& hi) {
  constexpr int n = LIST == 0 ? E8_NSTRICT : E8_NBOUNDARY;
  lo = hi = 0;
  if (idx >= n) return false;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int pl = LIST == 0 ? c_strict[idx][j] : c_boundary[idx][j];
    const int ph = LIST == 0 ? c_strict[idx][j + 4] : c_boundary[idx][j + 4];
    lo |= ((uint32_t)(4 * (pl - CMIN)) + wbyte) << (8 * j);
    hi |= ((uint32_t)(4 * (ph - CMIN)) + wbyte) << (8 * j);
  }
  return true;
}

struct Sel {
  uint32_t s[8];  // v_perm selectors (uniform): byte r_i of the candidate into byte 0
  uint32_t misc;  // sign bits, validity
};

__device__ __forceinline__ Sel read_sel(const Frame& F) {
  Sel o;
  const uint4 a = reinterpret_cast<const uint4*>(F.sel)[0];
  const uint4 b = reinterpret_cast<const uint4*>(F.sel)[1];
  o.s[0] = uniform(a.x); o.s[1] = uniform(a.y); o.s[2] = uniform(a.z); o.s[3] = uniform(a.w);
  o.s[4] = uniform(b.x); o.s[5] = uniform(b.y); o.s[6] = uniform(b.z); o.s[7] = uniform(b.w);
  o.misc = uniform(F.misc);
  return o;
}

// Recipe distance^2 of candidate (lo,hi): sum over original coordinates i, in
// order, of the per-query table entry (x_i - k_i)^2 (already fp32-rounded).
__device__ __forceinline__ float cand_d2(const float* qt, uint32_t lo, uint32_t hi, const Sel& sel) {
  float d = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float v = lds_f32(qt, __builtin_amdgcn_perm(hi, lo, sel.s[i]) + 256u * i);
    d = (i == 0) ? v : d + v;
  }
  return d;
}

__device__ __forceinline__ int32_t cand_slot(const uint32_t* st, uint32_t lo, uint32_t hi, const Sel& sel) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) m += lds_u32(st, __builtin_amdgcn_perm(hi, lo, sel.s[i]) + 256u * i);
  return (int32_t)(m >> 1);
}

// Lexicographic key of the lattice point itself (only consulted between equal
// (distance, location) pairs, which requires a torus side of 2).
__device__ __forceinline__ uint32_t cand_liftkey(uint32_t lo, uint32_t hi, const Sel& sel, const Frame& F) {
  uint32_t key = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t a = __builtin_amdgcn_perm(hi, lo, sel.s[i]);
    const int p = (int)((a & 63u) >> 2) + CMIN;
    const int c = F.c[i];
    const int k = ((sel.misc >> i) & 1u) ? c - p : c + p;
    key |= ((uint32_t)(k + 8) & 15u) << (4 * (7 - i));
  }
  return key;
}

template <int NS>
__device__ __forceinline__ int count_below(const uint32_t (&key)[NS], uint32_t t) {
  int c = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) c += __popcll(__ballot(key[s] < t));
  return c;
}

// Threshold selection of the closest ks (Sec. 2.6: ks = 32) over NS candidate
// slots per lane.  Returns the number selected; a slot is selected iff key < thr, or
// key == tie_key and it is among the `need` first of those in (location,
// lattice point) order (tie_key = KEY_INF when there is no tie).  *suspect is
// set when a point of the boundary list could enter the selection (the ks-th
// distance is within 1e-3 of the support edge, or fewer than ks points are in
// the support).
template <int NS>
__device__ __forceinline__ int threshold_k(const uint32_t (&key)[NS], const int ks, uint32_t& thr, uint32_t& tie_key,
                                           int& need, bool& suspect) {
  tie_key = KEY_INF;
  need = 0;
  const int n8 = count_below(key, KEY_8);
  if (n8 <= ks) {
    thr = KEY_8;
    suspect = true;
    return n8;
  }
  // bisection on the (monotone) bit patterns of non-negative floats:
  // invariant count(< lo) < ks < count(< hi)
  uint32_t lo_k = KEY_4, hi_k = KEY_8;
  int c = count_below(key, lo_k);
  if (c == ks) {
    thr = lo_k;
    suspect = false;
    return ks;
  }
  if (c > ks) {
    hi_k = lo_k;
    lo_k = 0;
  }
  while (hi_k - lo_k > 1) {
    const uint32_t mid = lo_k + ((hi_k - lo_k) >> 1);
    c = count_below(key, mid);
    if (c == ks) {
      thr = mid;
      suspect = mid > KEY_SUSPECT;
      return ks;
    }
    if (c < ks)
      lo_k = mid;
    else
      hi_k = mid;
  }
  // several candidates share the distance bits lo_k at the 32nd place
  thr = lo_k;
  tie_key = lo_k;
  need = ks - count_below(key, lo_k);
  suspect = lo_k > KEY_SUSPECT;
  return ks;
}

// Inclusive prefix sum across the 64 lanes of a wave (DPP row shifts, then row
// broadcasts to carry the row totals).
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, true);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, true);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, true);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, true);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xA, 0xF, false); // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xC, 0xF, false); // row_bcast:31
  return x;
}

// Threshold selection of the closest ks through a 64-bucket histogram of the
// distance bits on [4, 8) (bucket = top six mantissa bits): one LDS atomic per
// candidate, a wave prefix sum and one ballot locate the bucket of the ks-th
// point; the bisection then only runs inside that bucket.  Same contract as
// threshold_k.
template <int NS>
__device__ __forceinline__ int threshold_k_hist(const uint32_t (&key)[NS], uint32_t* hist, int lane, const int ks,
                                                uint32_t& thr, uint32_t& tie_key, int& need, bool& suspect) {
  const int clow = count_below(key, KEY_4);
  if (clow >= ks) return threshold_k<NS>(key, ks, thr, tie_key, need, suspect);  // never expected
  hist[lane] = 0;
  wave_lds_sync();
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (key[s] >= KEY_4 && key[s] < KEY_8) atomicAdd(&hist[(key[s] - KEY_4) >> 17], 1u);
  wave_lds_sync();
  const uint32_t h = hist[lane];
  const uint32_t pre = wave_inclusive_scan(h);
  const int n8 = clow + (int)__builtin_amdgcn_readlane(pre, 63);
  tie_key = KEY_INF;
  need = 0;
  if (n8 <= ks) {
    thr = KEY_8;
    suspect = true;
    return n8;
  }
  const uint64_t m = __ballot(clow + (int)pre >= ks);
  const int b = (int)__builtin_ctzll(m);
  const int below = clow + (int)__builtin_amdgcn_readlane(pre, b) - (int)__builtin_amdgcn_readlane(h, b);
  const int inb = (int)__builtin_amdgcn_readlane(h, b);
  uint32_t lo_k = KEY_4 + ((uint32_t)b << 17), hi_k = lo_k + (1u << 17);
  if (below + inb == ks) {
    thr = hi_k;
    suspect = hi_k > KEY_SUSPECT;
    return ks;
  }
  // invariant count(< lo) = below < ks < count(< hi)
  while (hi_k - lo_k > 1) {
    const uint32_t mid = lo_k + ((hi_k - lo_k) >> 1);
    const int c = count_below(key, mid);
    if (c == ks) {
      thr = mid;
      suspect = mid > KEY_SUSPECT;
      return ks;
    }
    if (c < ks)
      lo_k = mid;
    else
      hi_k = mid;
  }
  thr = lo_k;
  tie_key = lo_k;
  need = ks - count_below(key, lo_k);
  suspect = lo_k > KEY_SUSPECT;
  return ks;
}

template <int KS, int NBUF = 1>
struct Search {
  Tables& S;
  WaveLds<KS, NBUF>& W;
  int lane;
  uint32_t wbyte;
  uint32_t lo[NS_STRICT], hi[NS_STRICT];
  // lists of 64 and the untruncated lookup scan the boundary candidates often
  // (whenever the support holds fewer than 64 points) or always: they stay in
  // registers too (shorter lists read them from constant memory on the rare
  // path that needs them)
  static constexpr int NB_REG = KS >= 64 ? NS_BOUND : 1;
  uint32_t blo[NB_REG], bhi[NB_REG];
  // lane constants of the table build: coordinate i = lane/8, value v = lane%8
  int ti, tp, tK;
  uint32_t tS, tN0;
  uint32_t toff;  // byte offset of entry (i, w, v)

  // (the kernel argument is read field by field: holding a reference to it
  // would force the argument block into private memory)
  __device__ Search(const Params P, Tables& s, WaveLds<KS, NBUF>& wv, int w, int l)
      : S(s), W(wv), lane(l), wbyte(64u * (uint32_t)w) {
#pragma unroll
    for (int k = 0; k < NS_STRICT; ++k) load_candidate<0>(lane + WAVE * k, wbyte, lo[k], hi[k]);
    if constexpr (NB_REG == NS_BOUND) {
#pragma unroll
      for (int k = 0; k < NS_BOUND; ++k) load_candidate<1>(lane + WAVE * k, wbyte, blo[k], bhi[k]);
    }
    ti = lane >> 3;
    tp = (lane & 7) + CMIN;
    tK = P.K[0];
    tS = P.S[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) {
      tK = ti == i ? P.K[i] : tK;
      tS = ti == i ? P.S[i] : tS;
    }
    tN0 = ti == 0 ? P.N : 0u;
    toff = 256u * ti + wbyte + 4u * (lane & 7);
  }

  // Candidate (lo, hi) of lane-slot s: strict list in registers, boundary list
  // (only needed on the rare path) from constant memory.
  __device__ __forceinline__ void cand(int s, uint32_t& l, uint32_t& h) const {
    if (s < NS_STRICT) {
      l = lo[s];
      h = hi[s];
    } else if constexpr (NB_REG == NS_BOUND) {
      l = blo[s - NS_STRICT];
      h = bhi[s - NS_STRICT];
    } else {
      load_candidate<1>(lane + WAVE * (s - NS_STRICT), wbyte, l, h);
    }
  }

  // Per-query tables for frame F: entry (i, v) describes the lattice
  // coordinate k_i = c_i + s'_i (v + CMIN).
  __device__ __forceinline__ void build_tables(const Frame& F, uint32_t misc) {
    const float xi = F.x[ti];
    const int ci = F.c[ti];
    const int k = ((misc >> ti) & 1u) ? ci - tp : ci + tp;
    const float e = xi - (float)k;
    const float e2 = e * e;
    const int par = k & 1;
    int Y = (k - par) >> 1;
    // |x_i| < 2K, |x_i - c_i| <= 2 and |p| <= 4 put Y within [-K-3, K+3]: two
    // periods up or one down wrap it for K >= 4, K = 2 is a parity; the clamp
    // makes sure no rounding surprise can ever address outside the table
    Y += Y < 0 ? tK : 0;
    Y += Y < 0 ? tK : 0;
    Y -= Y >= tK ? tK : 0;
    Y = tK == 2 ? (Y & 1) : min(max(Y, 0), tK - 1);
    const uint32_t sl = (uint32_t)Y * tS + (par ? tN0 : 0u);
    *reinterpret_cast<float*>(reinterpret_cast<char*>(S.qt) + toff) = e2;
    *reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(S.st) + toff) = sl;
    *reinterpret_cast<float*>(reinterpret_cast<char*>(S.et) + toff) = e;
  }

  // Writes the selected candidates into W.nbr[buf][0..count) (slot-major, then
  // lane order); ties at the ks-th place are broken by (location, lattice point).
  template <int NS>
  __device__ __forceinline__ void emit(const uint32_t (&key)[NS], uint32_t thr, uint32_t tie_key, int need,
                                       const Sel& sel, const Frame& F, int buf) {
    int nt = 0;
    if (tie_key != KEY_INF) {
      // rare: list the tied candidates' (location, lattice point) keys (unrolled:
      // a runtime index into the candidate registers would spill them)
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const bool tied = key[s] == tie_key;
        const uint64_t m = __ballot(tied);
        if (m) {
          uint32_t l, h;
          cand(s, l, h);
          const int pos = nt + prefix_count(m);
          if (tied && pos < tie_max<KS>()) {
            W.tie[pos][0] = (uint32_t)cand_slot(S.st, l, h, sel);
            W.tie[pos][1] = cand_liftkey(l, h, sel, F);
          }
          nt += __popcll(m);
        }
      }
      nt = min(nt, tie_max<KS>());
      wave_lds_sync();
    }
    int base = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      bool p = key[s] < thr;
      if (tie_key != KEY_INF && key[s] == tie_key) {
        uint32_t l, h;
        cand(s, l, h);
        const uint32_t ms = (uint32_t)cand_slot(S.st, l, h, sel);
        const uint32_t mk = cand_liftkey(l, h, sel, F);
        int rank = 0;
#pragma unroll 1
        for (int e = 0; e < nt; ++e) {
          const uint32_t es = W.tie[e][0], ek = W.tie[e][1];
          rank += (es < ms || (es == ms && ek < mk)) ? 1 : 0;
        }
        p = rank < need;
      }
      const uint64_t m = __ballot(p);
      const int pos = base + prefix_count(m);
      if (p && pos < KS) {
        uint32_t l, h;
        cand(s, l, h);
        Nbr& n = W.nbr[buf][pos];
        n.lo = l;
        n.hi = h;
        n.dbits = key[s];
      }
      base += __popcll(m);
    }
  }

  // Full neighbour search of frame F into buffer `buf`: W.nbr[buf][0..KS) with
  // (lo, hi, dbits, slot) and W.wgt[buf] with the fp32 recipe weights, padded
  // with slot -1 / weight 0.  Returns the number of real neighbours.
  __device__ int run(const Frame& F, const Sel& sel, int buf) {
    int count = 0;
    if (sel.misc & 0x100u) {
      build_tables(F, sel.misc);
      wave_lds_sync();
      uint32_t thr = KEY_8, tie_key = KEY_INF;
      int need = 0;
      bool suspect = true;
      bool fast = false;
      // lists of up to 32: scan the E8_FAST2 candidates nearest to F first,
      // then the E8_FAST nearest; when the ks-th closest of a set is below
      // its bound none of the others can be among the closest ks (about 9 in
      // 10 queries take the first set, nearly every other the second)
      uint32_t key3[NS_FAST];
      if constexpr (KS <= NB) {
        uint32_t key2[NS_FAST2];
#pragma unroll
        for (int k = 0; k < NS_FAST2; ++k) key2[k] = key3[k] = __float_as_uint(cand_d2(S.qt, lo[k], hi[k], sel));
        count = threshold_k_hist<NS_FAST2>(key2, W.hist, lane, KS, thr, tie_key, need, suspect);
        fast = count == KS && !suspect && (tie_key != KEY_INF ? tie_key < KEY_FAST2 : thr <= KEY_FAST2);
        if (fast) {
          emit<NS_FAST2>(key2, thr, tie_key, need, sel, F, buf);
        } else {
#pragma unroll
          for (int k = NS_FAST2; k < NS_FAST; ++k) key3[k] = __float_as_uint(cand_d2(S.qt, lo[k], hi[k], sel));
          thr = KEY_8;
          tie_key = KEY_INF;
          need = 0;
          suspect = true;
          count = threshold_k_hist<NS_FAST>(key3, W.hist, lane, KS, thr, tie_key, need, suspect);
          fast = count == KS && !suspect && (tie_key != KEY_INF ? tie_key < KEY_FAST : thr <= KEY_FAST);
          if (fast) emit<NS_FAST>(key3, thr, tie_key, need, sel, F, buf);
        }
      }
      if (!fast) {
        uint32_t key[NS_STRICT];
#pragma unroll
        for (int k = 0; k < NS_STRICT; ++k) {
          if (KS <= NB && k < NS_FAST)
            key[k] = key3[k];
          else
            key[k] = (lane + WAVE * k < E8_NSTRICT) ? __float_as_uint(cand_d2(S.qt, lo[k], hi[k], sel)) : KEY_INF;
        }
        thr = KEY_8;
        tie_key = KEY_INF;
        need = 0;
        suspect = true;
        if constexpr (KS != KALL)
          count = threshold_k_hist<NS_STRICT>(key, W.hist, lane, KS, thr, tie_key, need, suspect);
        if (!suspect) {
          emit<NS_STRICT>(key, thr, tie_key, need, sel, F, buf);
        } else {
          // rare: rescan together with the points at distance exactly sqrt(8) from F
          uint32_t key7[NS_ALL];
#pragma unroll
          for (int k = 0; k < NS_STRICT; ++k) key7[k] = key[k];
          if constexpr (NB_REG == NS_BOUND) {
#pragma unroll
            for (int k = 0; k < NS_BOUND; ++k)
              key7[NS_STRICT + k] =
                  (lane + WAVE * k < E8_NBOUNDARY) ? __float_as_uint(cand_d2(S.qt, blo[k], bhi[k], sel)) : KEY_INF;
          } else {
#pragma unroll 1
            for (int k = 0; k < NS_BOUND; ++k) {
              uint32_t l, h;
              const bool okb = load_candidate<1>(lane + WAVE * k, wbyte, l, h);
              key7[NS_STRICT + k] = okb ? __float_as_uint(cand_d2(S.qt, l, h, sel)) : KEY_INF;
            }
          }
          if constexpr (KS == KALL) {
            // untruncated: every candidate whose recipe distance is below 8
            count = min(count_below(key7, KEY_8), KS);
            emit<NS_ALL>(key7, KEY_8, KEY_INF, 0, sel, F, buf);
          } else {
            bool suspect7;
            count = threshold_k<NS_ALL>(key7, KS, thr, tie_key, need, suspect7);
            emit<NS_ALL>(key7, thr, tie_key, need, sel, F, buf);
          }
        }
      }
      wave_lds_sync();
    }
    // locations and weights, one neighbour per lane
#pragma unroll
    for (int r = 0; r < (KS + WAVE - 1) / WAVE; ++r) {
      const int e = lane + WAVE * r;
      if (e < KS) {
        Nbr& n = W.nbr[buf][e];
        if (e < count) {
          n.slot = cand_slot(S.st, n.lo, n.hi, sel);
          const float u = 1.0f - __uint_as_float(n.dbits) * 0.125f;
          const float u2 = u * u;
          W.wgt[buf][e] = (u2 * u2) * F.s;  // exact for plain lookups (s = 1)
        } else {
          n.lo = n.hi = 0;
          n.dbits = KEY_INF;
          n.slot = -1;
          W.wgt[buf][e] = 0.0f;
        }
      }
    }
    wave_lds_sync();
    return count;
  }

  // The list of lookup l saved by the forward (NbrList), in place of run():
  // the per-query tables are rebuilt from the frame (the coordinate errors for
  // dq) and each entry's recipe distance is recomputed from its code exactly
  // as run() formed it.  Entries whose slot lies outside [0, N) count as
  // padding, so no list content can address outside the value table.
  __device__ int load(const Frame& F, const Sel& sel, int buf, const NbrList nl, int64_t l, uint32_t N) {
    static_assert(KS == NB, "saved lists hold the closest 32");
    const bool valid = (sel.misc & 0x100u) != 0;
    if (valid) {
      build_tables(F, sel.misc);
      wave_lds_sync();
    }
    bool real = false;
    if (lane < KS) {
      const size_t o = (size_t)l * KS + lane;
      const int32_t s = valid ? nl.slot[o] : -1;
      real = s >= 0 && (uint32_t)s < N;
      Nbr& n = W.nbr[buf][lane];
      if (real) {
        uint32_t l8, h8;
        bytes_of(nl.code[o] & 0xFFFFFFu, wbyte, l8, h8);
        n.lo = l8;
        n.hi = h8;
        n.dbits = __float_as_uint(cand_d2(S.qt, l8, h8, sel));
        n.slot = s;
        W.wgt[buf][lane] = nl.w[o];
      } else {
        n.lo = n.hi = 0;
        n.dbits = KEY_INF;
        n.slot = -1;
        W.wgt[buf][lane] = 0.0f;
      }
    }
    wave_lds_sync();
    return __popcll(__ballot(real));
  }

  // Writes list `buf` of lookup l to the saved lists (lanes 0..KS-1; nothing when !ok).
  __device__ __forceinline__ void save(int buf, const NbrList nl, int64_t l, bool ok) const {
    static_assert(KS == NB, "saved lists hold the closest 32");
    if (lane < KS && ok) {
      const size_t o = (size_t)l * KS + lane;
      const Nbr n = W.nbr[buf][lane];
      nl.slot[o] = n.slot;
      nl.w[o] = W.wgt[buf][lane];
      nl.code[o] = n.slot >= 0 ? code_of(n.lo, n.hi) : 0u;
    }
  }
};

// Input floats per lookup: q (8) or z (16, the activation layer).
template <bool TH>
constexpr int in_stride() { return TH ? 16 : 8; }

// Phase A for the wave's lookups [base, base + lpw).
template <bool TH>
__device__ __forceinline__ void phase_a(const float* __restrict__ in, int64_t base, int nl, const Params P,
                                        Frame* frames, int lane) {
  if (lane < nl) make_frame<TH>(in + (base + lane) * in_stride<TH>(), true, P, frames[lane]);
  wave_lds_sync();
}

// Same, for the lookups perm[base .. base + nl) of a reordered batch; returns
// this lane's lookup index (lane t holds the lookup of position base + t).  An
// index outside [0, L) (an order not written for these lookups) gets an empty
// list, and the kernels write nothing for it.
template <bool TH>
__device__ __forceinline__ uint32_t phase_a_perm(const float* __restrict__ in, const uint32_t* __restrict__ perm,
                                                 int64_t base, int nl, const Params P, Frame* frames, int lane) {
  uint32_t l = 0;
  if (lane < nl) {
    l = perm[base + lane];
    const bool ok = (int64_t)l < P.L;
    make_frame<TH>(in + (size_t)(ok ? l : 0u) * in_stride<TH>(), ok, P, frames[lane]);
  }
  wave_lds_sync();
  return l;
}

}  // namespace
