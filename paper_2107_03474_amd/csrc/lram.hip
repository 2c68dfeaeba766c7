// liblram -- LRAM lattice lookup for AMD Instinct MI355X (gfx950, CDNA4).
//
// Goucher & Troll, "Differentiable Random Access Memory using Lattices":
// lookup phi (Sec. 2.2) over the lattice Lambda = 2*E8 (Sec. 2.4) with the
// kernel f(r) = (1 - r^2/8)^4 (Sec. 2.5), truncated to the 32 closest points
// and found through the symmetry reduction of Sec. 2.6, plus its backward.
//
// Work decomposition (one wave = 64 lanes, up to 64 lookups per wave):
//   phase A  lane-per-lookup: wrap, E8 closest point (D8 and D8+1/2 decoders
//            with a parity fix), and the signed permutation that carries the
//            offset into the fundamental region F; the result (a 96-byte
//            "frame") goes to LDS.
//   phase B  wave-per-lookup: the wave builds three 8x8 per-query tables in LDS
//            (squared coordinate error, location contribution, coordinate
//            error) indexed by (original coordinate, candidate coordinate
//            value), scans the 232 candidate points of F (4 per lane) with one
//            v_perm + one LDS read per coordinate, selects the closest 32 (a
//            64-bucket histogram of the fp32 distance bits, then a ballot /
//            popcount bisection inside one bucket), and then gather-reduces
//            (forward) or scatters and forms dq (backward).  The row loads of
//            lookup t are in flight while the wave searches lookup t+1
//            (neighbour lists are double-buffered).
// The value-gradient scatter has three forms: row atomics, a location sort
// with a segmented reduction, and a per-batch merge of lookups ordered by
// their closest lattice point.  No MFMA: the path is a gather / scatter bound
// by HBM and by memory-side atomics, not a contraction.

#include <hip/hip_runtime.h>
#include <cmath>
#include <stdint.h>

#include <utility>

#include "../../include/lram.h"
#include "e8_candidates.inc"

namespace {

constexpr int NB = LRAM_NEIGHBOURS;  // 32, Sec. 2.6
constexpr int WAVE = 64;
constexpr int WAVES = 4;                 // waves per workgroup
constexpr int THREADS = WAVE * WAVES;
constexpr int NS_STRICT = (E8_NSTRICT + WAVE - 1) / WAVE;      // 4 candidate slots per lane
constexpr int NS_BOUND = (E8_NBOUNDARY + WAVE - 1) / WAVE;     // 3
constexpr int NS_ALL = NS_STRICT + NS_BOUND;
constexpr int CMIN = E8_CAND_MIN;
constexpr int NV = E8_CAND_MAX - E8_CAND_MIN + 1;
static_assert(NV == 8, "each per-query table row holds the 8 possible candidate coordinate values");
static_assert(WAVES <= 4, "the wave index is folded into byte-sized LDS offsets");
constexpr int KMAX = 8192;  // per-coordinate torus side bound: lattice coordinates fit in int16

// Candidates tied (equal fp32 distance bits) at the k-th place of a truncated
// list.  Large sets of equal distances inside the support arise only from the
// 240-point shell of a lattice point seen from a query a hair away from it
// along some offset d: the shell splits into groups of equal <p, d>, and the
// largest such group is the set of shell points orthogonal to one of them (an
// E7 root system, 126 points).  The untruncated list keeps no tie list.
template <int KS>
constexpr int tie_max() { return KS == 256 ? 1 : 128; }
// List width of the untruncated lookup (every point of the support).  The
// support is an open ball of radius sqrt 8; fp32 rounding of the distance
// recipe can admit points at distance exactly sqrt 8, so the count can pass
// the 121 of exact arithmetic, but a ball of that radius never holds more
// than the 1 + 240 points around a lattice point.
constexpr int KALL = 256;
constexpr uint32_t KEY_INF = 0x7F800000u;      // +inf: never selected
constexpr uint32_t KEY_8 = 0x41000000u;        // 8.0f: support boundary (open ball)
constexpr uint32_t KEY_4 = 0x40800000u;        // 4.0f: fewer than 32 points are ever closer
constexpr uint32_t KEY_SUSPECT = 0x40FFF7CFu;  // 7.999f

__constant__ signed char c_strict[E8_NSTRICT][8] = E8_STRICT_INIT;
__constant__ signed char c_boundary[E8_NBOUNDARY][8] = E8_BOUNDARY_INIT;

struct Params {
  int32_t K[8];
  uint32_t S[8];     // mixed-radix strides of the location map, S_7 = 1
  float twoK[8];     // torus side at the Lambda scale
  uint32_t N;
  int32_t lpw;       // lookups per wave (1..64)
  int64_t L;
  double cK[8];      // K_i / (2 pi): torus coordinate per radian of arg z_i (activation layer)
};

// Per-lookup frame written by phase A (96 bytes).
struct alignas(16) Frame {
  float x[8];         // Lambda-scale query, wrapped
  uint32_t sel[8];    // v_perm selector of original coordinate i: byte r_i (its F position) into byte 0
  int16_t c[8];       // closest lattice point
  uint32_t misc;      // bits 0-7: sign flips s'_i = -1; bit 8: query finite
  float s;            // output scale: 1, or (sum 1/|z_i|)^-1 behind the activation layer
  uint32_t pad[2];
};

// A selected neighbour as handed from the search to the gather / scatter.
struct alignas(16) Nbr {
  uint32_t lo, hi;    // packed candidate bytes (F coordinates)
  uint32_t dbits;     // fp32 recipe distance^2 bits
  int32_t slot;       // location, -1 for padding
};

// Per-wave search state for lists of KS neighbours.
template <int KS>
struct alignas(16) WaveLds {
  Nbr nbr[2][KS];     // double-buffered: lookup t+1 is searched while t is consumed
  float wgt[2][KS];
  uint32_t tie[tie_max<KS>()][2];
  uint32_t hist[64];  // distance histogram of the selection, 64 buckets on [4, 8)
};

// per-query tables, [coordinate i][wave w][value v] -> byte i*256 + w*64 + 4v
struct alignas(16) Tables {
  float qt[8 * 64];
  uint32_t st[8 * 64];
  float et[8 * 64];
};

// LDS of the search for FR lookups per wave and lists of KS neighbours.
template <int FR, int KS = NB>
struct alignas(16) SearchLds {
  Tables tab;
  WaveLds<KS> wave[WAVES];
  Frame frames[WAVES][FR];
};

__device__ __forceinline__ float lds_f32(const float* base, uint32_t byte_off) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(base) + byte_off);
}
__device__ __forceinline__ uint32_t lds_u32(const uint32_t* base, uint32_t byte_off) {
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(base) + byte_off);
}

__device__ __forceinline__ int prefix_count(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

__device__ __forceinline__ uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// Orders LDS traffic between lanes of one wave: the wave's LDS operations
// execute in issue order, so a compiler barrier is enough.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

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

// The query of one lookup and its output scale.  TH = false: q itself
// (8 floats), scale 1.  TH = true, the activation layer of Sec. 2.3: z_i =
// in[2i] + i in[2i+1], q_i = (K_i / 2 pi) arg z_i formed in fp64 and rounded
// once to fp32, scale (sum_i 1/|z_i|)^-1 (0 when some z_i = 0); a non-finite
// input gives a NaN query (empty neighbour list) and scale 0.
template <bool TH>
__device__ __forceinline__ void load_query(const float* __restrict__ in, const Params P, float (&qq)[8],
                                           float& scale) {
  if constexpr (!TH) {
    const float4 a = reinterpret_cast<const float4*>(in)[0];
    const float4 b = reinterpret_cast<const float4*>(in)[1];
    qq[0] = a.x; qq[1] = a.y; qq[2] = a.z; qq[3] = a.w;
    qq[4] = b.x; qq[5] = b.y; qq[6] = b.z; qq[7] = b.w;
    scale = 1.0f;
  } else {
    float z[16];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float4 v = reinterpret_cast<const float4*>(in)[k];
      z[4 * k] = v.x; z[4 * k + 1] = v.y; z[4 * k + 2] = v.z; z[4 * k + 3] = v.w;
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

template <int KS>
struct Search {
  Tables& S;
  WaveLds<KS>& W;
  int lane;
  uint32_t wbyte;
  uint32_t lo[NS_STRICT], hi[NS_STRICT];
  // lane constants of the table build: coordinate i = lane/8, value v = lane%8
  int ti, tp, tK;
  uint32_t tS, tN0;
  uint32_t toff;  // byte offset of entry (i, w, v)

  // (the kernel argument is read field by field: holding a reference to it
  // would force the argument block into private memory)
  __device__ Search(const Params P, Tables& s, WaveLds<KS>& wv, int w, int l)
      : S(s), W(wv), lane(l), wbyte(64u * (uint32_t)w) {
#pragma unroll
    for (int k = 0; k < NS_STRICT; ++k) load_candidate<0>(lane + WAVE * k, wbyte, lo[k], hi[k]);
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
      uint32_t key[NS_STRICT];
#pragma unroll
      for (int k = 0; k < NS_STRICT; ++k)
        key[k] = (lane + WAVE * k < E8_NSTRICT) ? __float_as_uint(cand_d2(S.qt, lo[k], hi[k], sel)) : KEY_INF;
      uint32_t thr = KEY_8, tie_key = KEY_INF;
      int need = 0;
      bool suspect = true;
      if constexpr (KS != KALL) count = threshold_k_hist<NS_STRICT>(key, W.hist, lane, KS, thr, tie_key, need, suspect);
      if (!suspect) {
        emit<NS_STRICT>(key, thr, tie_key, need, sel, F, buf);
      } else {
        // rare: rescan together with the points at distance exactly sqrt(8) from F
        uint32_t key7[NS_ALL];
#pragma unroll
        for (int k = 0; k < NS_STRICT; ++k) key7[k] = key[k];
#pragma unroll 1
        for (int k = 0; k < NS_BOUND; ++k) {
          uint32_t l, h;
          const bool okb = load_candidate<1>(lane + WAVE * k, wbyte, l, h);
          key7[NS_STRICT + k] = okb ? __float_as_uint(cand_d2(S.qt, l, h, sel)) : KEY_INF;
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
// this lane's lookup index (lane t holds the lookup of position base + t).
template <bool TH>
__device__ __forceinline__ uint32_t phase_a_perm(const float* __restrict__ in, const uint2* __restrict__ perm,
                                                 int64_t base, int nl, const Params P, Frame* frames, int lane) {
  uint32_t l = 0;
  if (lane < nl) {
    l = perm[base + lane].x;
    make_frame<TH>(in + (size_t)l * in_stride<TH>(), true, P, frames[lane]);
  }
  wave_lds_sync();
  return l;
}

// ---------------------------------------------------------------------------
// Kernels.

struct WaveCtx {
  int wave, lane;
  int64_t base;
  int nl;
};

__device__ __forceinline__ bool wave_ctx(const Params P, WaveCtx& c) {
  c.wave = threadIdx.x / WAVE;
  c.lane = threadIdx.x % WAVE;
  c.base = ((int64_t)blockIdx.x * WAVES + c.wave) * P.lpw;
  if (c.base >= P.L) return false;
  c.nl = (int)min<int64_t>(P.lpw, P.L - c.base);
  return true;
}

// Neighbour lists of width KS (NB = 32: Sec. 2.6; KALL: the whole support).
template <int KS>
__global__ void __launch_bounds__(THREADS) k_neighbors(const float* __restrict__ q, Params P,
                                                       int32_t* __restrict__ slot_out, float* __restrict__ w_out,
                                                       float* __restrict__ d2_out) {
  __shared__ SearchLds<WAVE, KS> S;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  Search<KS> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<KS>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<false>(q, c.base, c.nl, P, FR, c.lane);
  for (int t = 0; t < c.nl; ++t) {
    const Frame& F = FR[t];
    const Sel sel = read_sel(F);
    const int count = srch.run(F, sel, 0);
    const int64_t l = c.base + t;
    for (int me_i = c.lane; me_i < KS; me_i += WAVE) {
      // order the list by (distance bits, location, lattice point)
      const Nbr me = W.nbr[0][me_i];
      int rank = me_i;
      if (me_i < count) {
        const uint32_t mk = cand_liftkey(me.lo, me.hi, sel, F);
        rank = 0;
        for (int e = 0; e < count; ++e) {
          const Nbr o = W.nbr[0][e];
          bool less = o.dbits < me.dbits || (o.dbits == me.dbits && o.slot < me.slot);
          if (o.dbits == me.dbits && o.slot == me.slot && e != me_i) less = cand_liftkey(o.lo, o.hi, sel, F) < mk;
          rank += less ? 1 : 0;
        }
      }
      slot_out[l * KS + rank] = me.slot;
      w_out[l * KS + rank] = W.wgt[0][me_i];
      if (d2_out) d2_out[l * KS + rank] = __uint_as_float(me.dbits);
    }
    wave_lds_sync();
  }
}

// Row geometry of the backward's table reads for chunks of R rows.
template <int DT, int M, int R = NB>
struct RowGeom {
  static constexpr int ES = DT == LRAM_F32 ? 4 : 2;      // table element bytes
  static constexpr int RB = M * ES;                       // row bytes
  static constexpr int LPR = RB / 16;                     // lanes per row (16 B each)
  static constexpr int RPP = WAVE / LPR;                  // rows per pass
  static constexpr int NP = R / RPP;                      // passes
  static constexpr int EPC = 16 / ES;                     // elements per 16-byte chunk
  static_assert(RB % 16 == 0 && LPR <= WAVE && R % RPP == 0, "row geometry");
};

// Rows handled together by the gathers of a list of KS neighbours.
template <int KS>
constexpr int chunk_rows() { return KS < NB ? KS : NB; }

template <int DT, int EPC>
__device__ __forceinline__ void unpack16(const uint4 v, float (&f)[EPC]) {
  if constexpr (DT == LRAM_F32) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
  } else {
    f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
    f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
    f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
    f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
  }
}

// Gather geometry of the forward: each lane reads BPL contiguous bytes of a row,
// LPR lanes cover a row, one load instruction covers RPI rows, NI instructions
// cover the 32 rows; a lane accumulates EPL output elements over its NI rows and
// the RPI row groups are summed with xor shuffles.
template <int DT, int M, int R = NB>
struct FwdGeom {
  static constexpr int ES = DT == LRAM_F32 ? 4 : 2;
  static constexpr int RB = M * ES;
  static constexpr int BPL = (DT == LRAM_F32 && M == 64) ? 8 : 4;
  static constexpr int LPR = RB / BPL;
  static constexpr int RPI = WAVE / LPR;
  static constexpr int NI = R / RPI;
  static constexpr int EPL = BPL / ES;
  static constexpr int DW = BPL / 4;  // dwords per lane per row
  static_assert(LPR <= WAVE && WAVE % LPR == 0 && R % RPI == 0, "forward gather geometry");
};

// Loads the rows r0 .. r0 + R of list `buf` (R = the geometry's chunk).
template <int DT, int M, int KS, int R = NB>
__device__ __forceinline__ void fwd_issue(const char* __restrict__ tb, const WaveLds<KS>& W, int buf, int lane,
                                          uint32_t (&v)[FwdGeom<DT, M, R>::NI][FwdGeom<DT, M, R>::DW], int r0 = 0) {
  using G = FwdGeom<DT, M, R>;
  const int rsub = lane / G::LPR, col = lane % G::LPR;
#pragma unroll
  for (int p = 0; p < G::NI; ++p) {
    const int32_t s = W.nbr[buf][r0 + p * G::RPI + rsub].slot;
    const char* src = tb + (size_t)(s >= 0 ? s : 0) * G::RB + col * G::BPL;
    if constexpr (G::DW == 1) {
      v[p][0] = s >= 0 ? *reinterpret_cast<const uint32_t*>(src) : 0u;
    } else {
      const uint2 t = s >= 0 ? *reinterpret_cast<const uint2*>(src) : make_uint2(0, 0);
      v[p][0] = t.x;
      v[p][1] = t.y;
    }
  }
}

// acc += sum over the rows r0 .. r0 + R of w_j * v_j (this lane's columns).
template <int DT, int M, int KS, int R = NB>
__device__ __forceinline__ void fwd_accumulate(const WaveLds<KS>& W, int buf, int lane,
                                               const uint32_t (&v)[FwdGeom<DT, M, R>::NI][FwdGeom<DT, M, R>::DW],
                                               float (&acc)[FwdGeom<DT, M, R>::EPL], int r0 = 0) {
  using G = FwdGeom<DT, M, R>;
  const int rsub = lane / G::LPR;
#pragma unroll
  for (int p = 0; p < G::NI; ++p) {
    const float w = W.wgt[buf][r0 + p * G::RPI + rsub];
    if constexpr (DT == LRAM_F32) {
#pragma unroll
      for (int e = 0; e < G::EPL; ++e) acc[e] = fmaf(w, __uint_as_float(v[p][e]), acc[e]);
    } else {
#pragma unroll
      for (int d = 0; d < G::DW; ++d) {
        acc[2 * d] = fmaf(w, bf16_lo(v[p][d]), acc[2 * d]);
        acc[2 * d + 1] = fmaf(w, bf16_hi(v[p][d]), acc[2 * d + 1]);
      }
    }
  }
}

// Sums the row groups of the wave (xor shuffles) and writes out[l] once.
template <int DT, int M>
__device__ __forceinline__ void fwd_store(int lane, int64_t l, float (&acc)[FwdGeom<DT, M>::EPL],
                                          void* __restrict__ out) {
  using G = FwdGeom<DT, M>;
  const int rsub = lane / G::LPR, col = lane % G::LPR;
#pragma unroll
  for (int mask = G::LPR; mask < WAVE; mask <<= 1)
#pragma unroll
    for (int e = 0; e < G::EPL; ++e) acc[e] += __shfl_xor(acc[e], mask);
  if (rsub == 0) {
    char* ob = reinterpret_cast<char*>(out) + (size_t)l * G::RB + col * G::BPL;
    if constexpr (DT == LRAM_F32) {
      if constexpr (G::EPL == 1)
        *reinterpret_cast<float*>(ob) = acc[0];
      else
        *reinterpret_cast<float2*>(ob) = make_float2(acc[0], acc[1]);
    } else {
      *reinterpret_cast<uint32_t*>(ob) = pack_bf16x2(acc[0], acc[1]);
    }
  }
}

template <int DT, int M>
__device__ __forceinline__ void fwd_consume(const WaveLds<NB>& W, int buf, int lane, int64_t l,
                                            const uint32_t (&v)[FwdGeom<DT, M>::NI][FwdGeom<DT, M>::DW],
                                            void* __restrict__ out) {
  float acc[FwdGeom<DT, M>::EPL];
#pragma unroll
  for (int e = 0; e < FwdGeom<DT, M>::EPL; ++e) acc[e] = 0.0f;
  fwd_accumulate<DT, M, NB>(W, buf, lane, v, acc);
  fwd_store<DT, M>(lane, l, acc, out);
}

// TH: the input is the activation layer's z [L][16] instead of q [L][8]; the
// scale s is folded into the weights by the search.
template <int DT, int M, bool TH>
__global__ void __launch_bounds__(THREADS) k_forward(const float* __restrict__ q, Params P,
                                                     const void* __restrict__ table, void* __restrict__ out) {
  using G = FwdGeom<DT, M>;
  __shared__ SearchLds<WAVE> S;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  Search<NB> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<NB>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<TH>(q, c.base, c.nl, P, FR, c.lane);
  const char* tb = reinterpret_cast<const char*>(table);
  uint32_t v[G::NI][G::DW];
  srch.run(FR[0], read_sel(FR[0]), 0);
  fwd_issue<DT, M, NB>(tb, W, 0, c.lane, v);
  for (int t = 0; t < c.nl; ++t) {
    const int buf = t & 1;
    // search lookup t+1 while the rows of lookup t are in flight
    if (t + 1 < c.nl) srch.run(FR[t + 1], read_sel(FR[t + 1]), buf ^ 1);
    fwd_consume<DT, M>(W, buf, c.lane, c.base + t, v, out);
    if (t + 1 < c.nl) fwd_issue<DT, M, NB>(tb, W, buf ^ 1, c.lane, v);
  }
}

// Forward with lists of KS != 32 neighbours (the variable-k and untruncated
// lookups): per lookup, the rows are gathered in chunks of up to 32, only as
// many chunks as the lookup has neighbours.
template <int DT, int M, int KS>
__global__ void __launch_bounds__(THREADS) k_forward_k(const float* __restrict__ q, Params P,
                                                       const void* __restrict__ table, void* __restrict__ out) {
  constexpr int R = chunk_rows<KS>();
  using G = FwdGeom<DT, M, R>;
  __shared__ SearchLds<WAVE, KS> S;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  Search<KS> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<KS>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<false>(q, c.base, c.nl, P, FR, c.lane);
  const char* tb = reinterpret_cast<const char*>(table);
  for (int t = 0; t < c.nl; ++t) {
    const int count = srch.run(FR[t], read_sel(FR[t]), 0);
    float acc[G::EPL];
#pragma unroll
    for (int e = 0; e < G::EPL; ++e) acc[e] = 0.0f;
    for (int r0 = 0; r0 < count; r0 += R) {
      uint32_t v[G::NI][G::DW];
      fwd_issue<DT, M, KS, R>(tb, W, 0, c.lane, v, r0);
      fwd_accumulate<DT, M, KS, R>(W, 0, c.lane, v, acc, r0);
    }
    fwd_store<DT, M>(c.lane, c.base + t, acc, out);
    wave_lds_sync();
  }
}

// The merged scatter pays off when lookups share their closest lattice point
// (their neighbour lists then overlap): it is chosen when at least a tenth of
// the lookups share theirs with another lookup of the batch.
__device__ __forceinline__ bool merge_chosen(uint32_t shared, int64_t L) { return 10 * (int64_t)shared >= L; }

// Backward, fused with the query gradient: per lookup, read the 32 rows once
// for <G, v_j> and form dq from the coordinate errors.

// Value-gradient scatter of one lookup: M consecutive lanes own one gradient
// row, so each atomic instruction covers 64/M whole rows.
template <int M, int KS>
__device__ __forceinline__ void scatter_atomic(const WaveLds<KS>& W, int count, const float* __restrict__ gout,
                                               int64_t l, float* __restrict__ gtab, int lane) {
  constexpr int RA = WAVE / M;
  const int col = lane % M;
  const float gc = gout[(size_t)l * M + col];
  const int kend = KS == NB ? NB / RA : (min(count, KS) + RA - 1) / RA;
#pragma unroll 4
  for (int k = 0; k < kend; ++k) {
    const int j = k * RA + lane / M;
    const int32_t s = W.nbr[0][j].slot;
    if (s >= 0) unsafeAtomicAdd(gtab + (size_t)s * M + col, W.wgt[0][j] * gc);
  }
}

// dq_i = sum_j -2 u_j^3 (x_i - k_{j,i}) <G, v_j> of one lookup (zero without
// neighbours), written to gq[l][8].
// TH (activation layer): also dL/ds = sum_j w_j <G, v_j> = <G, phi>, and the
// chain through q_i = c_i arg z_i and s = (sum 1/|z_i|)^-1 (Sec. 2.3), with
// dL/dq = s dq:
//   dL/da_i = dL/ds s^2 a_i / r_i^3 - dL/dq_i c_i b_i / r_i^2,
//   dL/db_i = dL/ds s^2 b_i / r_i^3 + dL/dq_i c_i a_i / r_i^2,
// written to gq[l][16] (zero where s = 0); zin is z.
template <int DT, int M, bool TH, int KS>
__device__ __forceinline__ void grad_query(const Frame& F, const WaveLds<KS>& W, const Tables& T, int count,
                                           const char* __restrict__ tb, const float* __restrict__ gout, int64_t l,
                                           int lane, float* __restrict__ gq, const float* __restrict__ zin,
                                           const Params& P) {
  constexpr int R = chunk_rows<KS>();  // rows per chunk of the row loop
  using G = RowGeom<DT, M, R>;
  constexpr int ICOORD = G::LPR >= 8 ? 1 : 8 / G::LPR;  // query coordinates per lane
  const int rsub = lane / G::LPR, ch = lane % G::LPR;
  double dq[ICOORD];
  double dls = 0.0;  // dL/ds (TH)
#pragma unroll
  for (int k = 0; k < ICOORD; ++k) dq[k] = 0.0;
  if (count > 0) {
    float g[G::EPC];
    const float* gp = gout + (size_t)l * M + ch * G::EPC;
#pragma unroll
    for (int e = 0; e < G::EPC; e += 4) {
      const float4 gv = *reinterpret_cast<const float4*>(gp + e);
      g[e] = gv.x; g[e + 1] = gv.y; g[e + 2] = gv.z; g[e + 3] = gv.w;
    }
    // per-lane selectors of the query coordinates this lane accumulates
    uint32_t lsel[ICOORD];
#pragma unroll
    for (int k = 0; k < ICOORD; ++k) {
      lsel[k] = F.sel[(ch + k * G::LPR) & 7];
    }
    for (int r0 = 0; r0 < (KS == NB ? 1 : count); r0 += R) {
    uint4 v[G::NP];
    int32_t sl[G::NP];
#pragma unroll
    for (int p = 0; p < G::NP; ++p) {
      sl[p] = W.nbr[0][r0 + p * G::RPP + rsub].slot;
      v[p] = sl[p] >= 0 ? *reinterpret_cast<const uint4*>(tb + (size_t)sl[p] * G::RB + ch * 16)
                        : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int p = 0; p < G::NP; ++p) {
      const int j = r0 + p * G::RPP + rsub;
      float f[G::EPC];
      unpack16<DT, G::EPC>(v[p], f);
      // <G, v_j>: this lane's chunk, then a sum over the LPR lanes of the row,
      // in fp64 (fp32 x fp32 products are exact there).  Next to a lattice
      // point one term carries all of dq (and behind the activation layer
      // dL/ds is sum_j w_j <G, v_j>), so a cancelling fp32 dot product would
      // become the relative error of the whole gradient.
      double pd64 = 0.0;
#pragma unroll
      for (int e = 0; e < G::EPC; ++e) pd64 = fma((double)g[e], (double)f[e], pd64);
#pragma unroll
      for (int mask = 1; mask < G::LPR; mask <<= 1) pd64 += __shfl_xor(pd64, mask);
      if (sl[p] >= 0) {
        const Nbr n = W.nbr[0][j];
        const float u = 1.0f - __uint_as_float(n.dbits) * 0.125f;
        const double a = -2.0 * (double)(u * u * u) * pd64;
        if constexpr (TH) {
          const float u2 = u * u;
          dls = fma((double)(u2 * u2), pd64, dls);
        }
#pragma unroll
        for (int k = 0; k < ICOORD; ++k) {
          const int i = ch + k * G::LPR;
          if (i < 8) {
            const uint32_t ab = __builtin_amdgcn_perm(n.hi, n.lo, lsel[k]);
            dq[k] = fma(a, (double)lds_f32(T.et, ab + 256u * i), dq[k]);
          }
        }
      }
    }
    }  // chunks of R rows
  }
#pragma unroll
  for (int mask = G::LPR; mask < WAVE; mask <<= 1) {
#pragma unroll
    for (int k = 0; k < ICOORD; ++k) dq[k] += __shfl_xor(dq[k], mask);
    if constexpr (TH) dls += __shfl_xor(dls, mask);
  }
  if (rsub == 0) {
#pragma unroll
    for (int k = 0; k < ICOORD; ++k) {
      const int i = ch + k * G::LPR;
      if (i >= 8) continue;
      if constexpr (!TH) {
        gq[l * 8 + i] = (float)dq[k];
      } else {
        double ci = P.cK[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) ci = i == e ? P.cK[e] : ci;
        const double sc = F.s;
        double ga = 0.0, gb = 0.0;
        if (sc > 0.0) {
          const float2 ab = *reinterpret_cast<const float2*>(zin + l * 16 + 2 * i);
          const double a = ab.x, b = ab.y;
          const double r2 = a * a + b * b;
          const double r3 = r2 * sqrt(r2);
          const double ds = dls * sc * sc, dqs = dq[k] * sc * ci;
          ga = ds * a / r3 - dqs * b / r2;
          gb = ds * b / r3 + dqs * a / r2;
        }
        *reinterpret_cast<float2*>(gq + l * 16 + 2 * i) = make_float2((float)ga, (float)gb);
      }
    }
  }
}

// The value gradient is either added straight into grad_table with fp32
// atomics (EMIT = false), or emitted as (location, (lookup, w_j)) pairs for
// the sorted segmented reduction (EMIT = true; padding gets the key N, which
// sorts last).
// gate (nullable): the merged scatter's device-side choice -- this kernel does
// nothing when the batch is merged instead (see merge_chosen).
template <int DT, int M, bool EMIT, bool TH, int KS = NB>
__global__ void __launch_bounds__(THREADS) k_backward(const float* __restrict__ q, Params P,
                                                      const void* __restrict__ table,
                                                      const float* __restrict__ gout, float* __restrict__ gtab,
                                                      float* __restrict__ gq, uint32_t* __restrict__ pair_key,
                                                      uint2* __restrict__ pair_val, const uint32_t* __restrict__ gate) {
  static_assert(!EMIT || KS == NB, "the sorted scatter takes lists of 32");
  __shared__ SearchLds<WAVE, KS> S;
  if (gate && merge_chosen(*gate, P.L)) return;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  const int lane = c.lane;
  Search<KS> srch(P, S.tab, S.wave[c.wave], c.wave, lane);
  WaveLds<KS>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<TH>(q, c.base, c.nl, P, FR, lane);
  const char* tb = reinterpret_cast<const char*>(table);
  for (int t = 0; t < c.nl; ++t) {
    const Frame& F = FR[t];
    const Sel sel = read_sel(F);
    const int count = srch.run(F, sel, 0);
    const int64_t l = c.base + t;
    if (!EMIT && gtab && count > 0) scatter_atomic<M, KS>(W, count, gout, l, gtab, lane);
    if (gq) grad_query<DT, M, TH, KS>(F, W, S.tab, count, tb, gout, l, lane, gq, q, P);
    if (EMIT && gtab && lane < NB) {
      const int32_t s = W.nbr[0][lane].slot;
      pair_key[l * NB + lane] = s >= 0 ? (uint32_t)s : P.N;
      pair_val[l * NB + lane] = make_uint2((uint32_t)l, __float_as_uint(W.wgt[0][lane]));
    }
    wave_lds_sync();
  }
}

// Sorted value-gradient scatter: a stable LSD radix sort of the (location,
// (lookup, weight)) pairs by location, then a segmented reduction that writes
// every touched gradient row with one read-modify-write.

constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;
constexpr int SORT_ROUNDS = 16;                    // elements per thread per tile
constexpr int SORT_TILE = THREADS * SORT_ROUNDS;   // 4096
constexpr int SCAN_TILE = THREADS * 16;            // 4096 entries per scan block

// hist[d * nblocks + b] = number of keys in tile b whose digit is d
__global__ void __launch_bounds__(THREADS) k_radix_hist(const uint32_t* __restrict__ keys, int64_t n, int shift,
                                                        uint32_t* __restrict__ hist, int nblocks) {
  __shared__ uint32_t h[RADIX];
  const int t = threadIdx.x;
  h[t] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
#pragma unroll 4
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int64_t i = base + r * THREADS + t;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & (RADIX - 1)], 1u);
  }
  __syncthreads();
  hist[(int64_t)t * nblocks + blockIdx.x] = h[t];
}

// Exclusive scan, three kernels: per-block scan with block totals, scan of the
// totals (one block), add the scanned totals back.
__global__ void __launch_bounds__(THREADS) k_scan_blocks(uint32_t* __restrict__ a, int64_t n,
                                                         uint32_t* __restrict__ totals) {
  __shared__ uint32_t part[THREADS];
  const int t = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + (int64_t)t * 16;
  uint32_t v[16];
  uint32_t sum = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    v[k] = base + k < n ? a[base + k] : 0u;
    sum += v[k];
  }
  part[t] = sum;
  __syncthreads();
  for (int off = 1; off < THREADS; off <<= 1) {
    const uint32_t x = t >= off ? part[t - off] : 0u;
    __syncthreads();
    part[t] += x;
    __syncthreads();
  }
  uint32_t run = part[t] - sum;  // exclusive prefix of this thread's 16 entries
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    if (base + k < n) a[base + k] = run;
    run += v[k];
  }
  if (t == THREADS - 1) totals[blockIdx.x] = part[t];
}

__global__ void __launch_bounds__(THREADS) k_scan_totals(uint32_t* __restrict__ totals, int64_t n) {
  __shared__ uint32_t part[THREADS];
  __shared__ uint32_t carry;
  const int t = threadIdx.x;
  if (t == 0) carry = 0;
  __syncthreads();
  for (int64_t base = 0; base < n; base += THREADS) {
    const uint32_t v = base + t < n ? totals[base + t] : 0u;
    part[t] = v;
    __syncthreads();
    for (int off = 1; off < THREADS; off <<= 1) {
      const uint32_t x = t >= off ? part[t - off] : 0u;
      __syncthreads();
      part[t] += x;
      __syncthreads();
    }
    if (base + t < n) totals[base + t] = carry + part[t] - v;
    __syncthreads();
    if (t == THREADS - 1) carry += part[t];
    __syncthreads();
  }
}

__global__ void __launch_bounds__(THREADS) k_scan_add(uint32_t* __restrict__ a, int64_t n,
                                                      const uint32_t* __restrict__ totals) {
  const uint32_t add = totals[blockIdx.x];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
#pragma unroll 4
  for (int k = 0; k < 16; ++k) {
    const int64_t i = base + k * THREADS + threadIdx.x;
    if (i < n) a[i] += add;
  }
}

// Stable scatter of one radix pass.  Element order inside a tile is (round,
// wave, lane), i.e. index order; ranks among equal digits come from an 8-ballot
// match inside the wave plus per-(wave, digit) counts carried across rounds.
// The tile is first ordered by digit in LDS (a 2-byte permutation), then
// written out in that order so that consecutive threads store consecutive
// addresses of a digit's output run.
__global__ void __launch_bounds__(THREADS) k_radix_scatter(const uint32_t* __restrict__ kin,
                                                           const uint2* __restrict__ vin, int64_t n, int shift,
                                                           const uint32_t* __restrict__ offs, int nblocks,
                                                           uint32_t* __restrict__ kout, uint2* __restrict__ vout) {
  __shared__ uint32_t run_cnt[RADIX];
  __shared__ uint32_t wave_cnt[WAVES][RADIX];
  __shared__ uint32_t tile_start[RADIX];
  __shared__ uint32_t glob_off[RADIX];
  __shared__ uint16_t perm[SORT_TILE];
  const int t = threadIdx.x, w = t / WAVE, lane = t % WAVE;
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
  const int cnt = (int)min<int64_t>(SORT_TILE, n - base);
  // tile histogram, then its exclusive prefix (tile-local start of each digit)
  run_cnt[t] = 0;
  __syncthreads();
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = r * THREADS + t;
    if (j < cnt) atomicAdd(&run_cnt[(kin[base + j] >> shift) & (RADIX - 1)], 1u);
  }
  __syncthreads();
  const uint32_t c = run_cnt[t];
  wave_cnt[0][t] = c;
  __syncthreads();
  for (int off = 1; off < RADIX; off <<= 1) {
    const uint32_t x = t >= off ? wave_cnt[0][t - off] : 0u;
    __syncthreads();
    wave_cnt[0][t] += x;
    __syncthreads();
  }
  tile_start[t] = wave_cnt[0][t] - c;
  run_cnt[t] = wave_cnt[0][t] - c;
  glob_off[t] = offs[(int64_t)t * nblocks + blockIdx.x];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < WAVES; ++k) wave_cnt[k][t] = 0;
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (WAVE - lane));
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = r * THREADS + t;
    const bool valid = j < cnt;
    const uint32_t key = valid ? kin[base + j] : 0u;
    const uint32_t d = (key >> shift) & (RADIX - 1);
    uint64_t match = __ballot(valid);
#pragma unroll
    for (int b = 0; b < RADIX_BITS; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      match &= bit ? bb : ~bb;
    }
    const int rank = __popcll(match & lt);
    if (valid && rank == 0) wave_cnt[w][d] = (uint32_t)__popcll(match);
    __syncthreads();
    {
      uint32_t run = run_cnt[t];
#pragma unroll
      for (int k = 0; k < WAVES; ++k) {
        const uint32_t cw = wave_cnt[k][t];
        wave_cnt[k][t] = run;
        run += cw;
      }
      run_cnt[t] = run;
    }
    __syncthreads();
    if (valid) perm[wave_cnt[w][d] + (uint32_t)rank] = (uint16_t)j;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < WAVES; ++k) wave_cnt[k][t] = 0;
    __syncthreads();
  }
  // write out in digit order (the tile's inputs are still in cache)
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = r * THREADS + t;
    if (j < cnt) {
      const int src = perm[j];
      const uint32_t key = kin[base + src];
      const uint32_t d = (key >> shift) & (RADIX - 1);
      const uint32_t pos = glob_off[d] + (uint32_t)j - tile_start[d];
      kout[pos] = key;
      vout[pos] = vin[base + src];
    }
  }
}

// Segmented reduction of the sorted pairs.  A group of M lanes (lane = column
// of the gradient row) owns a span of consecutive pairs (256, fewer for small
// batches so that every CU gets work) and walks it in
// order, prefetching 16 pairs and their upstream-gradient rows at a time; it
// accumulates w * G[lookup] while the location stays the same and writes each
// finished run of one location with a single plain read-modify-write when the
// run lies inside the span (no other group touches that row), or with fp32
// atomics for the runs cut by the span edges (so a hot location costs one
// atomic row per span of updates and never serialises one group).
constexpr int SEG_SPAN = 256;
constexpr int SEG_BATCH = 16;

template <int M>
__device__ __forceinline__ void seg_flush(float* __restrict__ gtab, uint32_t key, int col, float acc, bool plain) {
  float* dst = gtab + (size_t)key * M + col;
  if (plain)
    *dst += acc;
  else
    unsafeAtomicAdd(dst, acc);
}

template <int M>
__global__ void __launch_bounds__(THREADS) k_segreduce(const uint32_t* __restrict__ keys,
                                                       const uint2* __restrict__ vals, int64_t n, uint32_t N,
                                                       const float* __restrict__ gout, float* __restrict__ gtab,
                                                       int span) {
  const int64_t group = ((int64_t)blockIdx.x * THREADS + threadIdx.x) / M;
  const int col = threadIdx.x % M;
  const int64_t b = group * span;
  if (b >= n) return;
  const int64_t e = min<int64_t>(n, b + span);
  uint32_t cur = keys[b];
  if (cur >= N) return;  // padding sorts last
  bool head_here = (b == 0) || keys[b - 1] != cur;
  float acc = 0.0f;
  bool pad = false;  // reached the padding (key N), which sorts last
  for (int64_t p = b; p < e && !pad; p += SEG_BATCH) {
    uint32_t k[SEG_BATCH];
    float wv[SEG_BATCH], g[SEG_BATCH];
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      const int64_t q = p + u;
      k[u] = q < e ? keys[q] : N;
      const uint2 v = q < e ? vals[q] : make_uint2(0, 0);
      wv[u] = __uint_as_float(v.y);
      g[u] = k[u] < N ? gout[(size_t)v.x * M + col] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      if (p + u < e && !pad) {
        if (k[u] >= N) {
          pad = true;  // the current run ended just before the padding
        } else {
          if (k[u] != cur) {
            seg_flush<M>(gtab, cur, col, acc, head_here);  // ended inside the span
            cur = k[u];
            acc = 0.0f;
            head_here = true;
          }
          acc = fmaf(wv[u], g[u], acc);
        }
      }
    }
  }
  if (pad) {
    seg_flush<M>(gtab, cur, col, acc, head_here);
    return;
  }
  // the span's last run: plain only if it also ends inside the span
  const bool ends_here = (e == n) || keys[e] != cur;
  seg_flush<M>(gtab, cur, col, acc, head_here && ends_here);
}

// ---------------------------------------------------------------------------
// Batch-merged scatter.  Lookups whose queries share the closest lattice point
// share most of their 32 neighbours; the lookups are ordered by that point's
// location (radix sort above), the backward emits (location, w) pairs in that
// order, and each batch of MERGE_T consecutive lookups is reduced in LDS to one
// fp32 atomic row per distinct location of the batch.

// key[l] = location of the closest point of Lambda to q_l (N for a non-finite
// query), val[l] = (l, 0).
template <bool TH>
__global__ void __launch_bounds__(THREADS) k_cell_key(const float* __restrict__ q, Params P,
                                                      uint32_t* __restrict__ key, uint2* __restrict__ val) {
  const int64_t l = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (l >= P.L) return;
  float x[8], qq[8], scale;
  int c[8];
  load_query<TH>(q + l * in_stride<TH>(), P, qq, scale);
  const bool valid = closest_point(qq, true, P, x, c);
  uint32_t loc = P.N;
  if (valid) {
    const int eps = c[0] & 1;
    uint32_t acc = eps ? P.N : 0u;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int y = (c[i] - eps) >> 1;  // in [-1, K_i]
      y = y < 0 ? y + P.K[i] : (y >= P.K[i] ? y - P.K[i] : y);
      acc += (uint32_t)y * P.S[i];
    }
    loc = acc >> 1;
  }
  key[l] = loc;
  val[l] = make_uint2((uint32_t)l, 0u);
}

// Activation layer coordinates: q[l] (8 fp32) and scale s[l] as the lookups see them.
__global__ void __launch_bounds__(THREADS) k_theta_coords(const float* __restrict__ z, Params P,
                                                          float* __restrict__ q, float* __restrict__ s) {
  const int64_t l = (int64_t)blockIdx.x * THREADS + threadIdx.x;
  if (l >= P.L) return;
  float qq[8], scale;
  load_query<true>(z + l * 16, P, qq, scale);
  reinterpret_cast<float4*>(q + l * 8)[0] = make_float4(qq[0], qq[1], qq[2], qq[3]);
  reinterpret_cast<float4*>(q + l * 8)[1] = make_float4(qq[4], qq[5], qq[6], qq[7]);
  if (s) s[l] = scale;
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint32_t v) {
  if (threadIdx.x == 0) *p = v;
}

// *count += number of positions whose sorted key equals a neighbour's.
__global__ void __launch_bounds__(THREADS) k_count_shared(const uint32_t* __restrict__ keys, int64_t L,
                                                          uint32_t* __restrict__ count) {
  uint32_t c = 0;
  for (int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x; i < L; i += (int64_t)gridDim.x * THREADS) {
    const uint32_t k = keys[i];
    c += ((i > 0 && keys[i - 1] == k) || (i + 1 < L && keys[i + 1] == k)) ? 1u : 0u;
  }
#pragma unroll
  for (int mask = 1; mask < WAVE; mask <<= 1) c += __shfl_xor(c, mask);
  if (threadIdx.x % WAVE == 0 && c) atomicAdd(count, c);
}

constexpr int64_t AUTO_MERGE_MIN = 131072;      // LRAM_SCATTER_AUTO merges from this many lookups on
constexpr int MERGE_T = 64;                     // lookups per batch (one workgroup)
constexpr int MERGE_LPW = MERGE_T / WAVES;      // lookups per wave
constexpr int MERGE_P = MERGE_T * NB;           // pairs per batch
constexpr int MERGE_H = 2 * MERGE_P;            // hash entries (load factor <= 1/2)
constexpr int MERGE_HBITS = 12;
static_assert((1 << MERGE_HBITS) == MERGE_H, "hash size");
constexpr int MERGE_PPT = MERGE_P / THREADS;    // pairs per thread
constexpr int MERGE_HPT = MERGE_H / THREADS;    // hash entries per thread (consecutive)
constexpr int32_t MERGE_EMPTY = -1;
static_assert(MERGE_T <= 256 && MERGE_P < 65536, "batch-local indices are 8 and 16 bits wide");

template <int M>
struct alignas(16) MergeWork {
  int32_t tag[MERGE_H];         // location of each hash entry; later pair weights and lookups in group order
  uint32_t cnt[MERGE_H / 2];    // 16-bit pair count of each entry, then its first position in group order
  float g[MERGE_T][M];          // upstream gradient rows of the batch
  uint32_t wsum[WAVES][2];
  uint32_t ngroups;
};

template <int M>
struct alignas(16) FusedLds {
  union {
    struct {
      int32_t loc[MERGE_P];     // (location, w) of every pair, [lookup in batch][j]
      float w[MERGE_P];
    } pairs;
    struct {
      int32_t loc[MERGE_P];     // distinct locations of the batch
      uint16_t start[MERGE_P + 2];  // first position of each location's pairs in group order
    } grp;
  } a;
  union {
    SearchLds<MERGE_LPW> search;
    MergeWork<M> merge;
  } b;
};

// One workgroup = one batch of MERGE_T consecutive positions of the order
// perm: each wave searches MERGE_LPW lookups (with dq as in k_backward) and
// leaves their (location, w) pairs in LDS; then the workgroup hashes the
// pairs by location, lays them out grouped by location, and M lanes per
// distinct location sum w * G over its pairs and add the row with fp32 atomics.
// Several workgroups per CU overlap one's search with another's atomics.
// A batch in which fewer than a tenth of the lookups share their closest
// point with a neighbour in the order (queries spread thinly over the torus)
// has little to merge: it scatters with per-lookup atomics instead.
template <int DT, int M, bool TH>
__global__ void __launch_bounds__(THREADS) k_backward_merged(const float* __restrict__ q, Params P,
                                                             const void* __restrict__ table,
                                                             const float* __restrict__ gout,
                                                             float* __restrict__ gtab, float* __restrict__ gq,
                                                             const uint32_t* __restrict__ skey,
                                                             const uint2* __restrict__ perm,
                                                             const uint32_t* __restrict__ gate) {
  __shared__ FusedLds<M> S;
  if (!merge_chosen(*gate, P.L)) return;  // the batch is scattered by k_backward instead
  const int t = threadIdx.x, wave = t / WAVE, lane = t % WAVE;
  const int64_t bbase = (int64_t)blockIdx.x * (WAVES * P.lpw);
  const int nt = (int)min<int64_t>(WAVES * P.lpw, P.L - bbase);
  bool shared = false;
  if (t < nt) {
    const uint32_t k = skey[bbase + t];
    shared = (t > 0 && skey[bbase + t - 1] == k) || (t + 1 < nt && skey[bbase + t + 1] == k);
  }
  const bool merge = 10 * __syncthreads_count(shared) >= nt;
  {
    const int64_t base = bbase + (int64_t)wave * P.lpw;
    const int nl = (int)max<int64_t>(0, min<int64_t>(P.lpw, P.L - base));
    if (nl > 0) {
      Search<NB> srch(P, S.b.search.tab, S.b.search.wave[wave], wave, lane);
      WaveLds<NB>& W = S.b.search.wave[wave];
      Frame* FR = S.b.search.frames[wave];
      const uint32_t my_l = phase_a_perm<TH>(q, perm, base, nl, P, FR, lane);
      const char* tb = reinterpret_cast<const char*>(table);
      for (int i = 0; i < nl; ++i) {
        const Frame& F = FR[i];
        const Sel sel = read_sel(F);
        const int count = srch.run(F, sel, 0);
        const int64_t l = (int64_t)__builtin_amdgcn_readlane(my_l, i);
        if (!merge && count > 0) scatter_atomic<M, NB>(W, count, gout, l, gtab, lane);
        if (gq) grad_query<DT, M, TH, NB>(F, W, S.b.search.tab, count, tb, gout, l, lane, gq, q, P);
        if (merge && lane < NB) {
          const int pidx = (wave * P.lpw + i) * NB + lane;
          S.a.pairs.loc[pidx] = W.nbr[0][lane].slot;
          S.a.pairs.w[pidx] = W.wgt[0][lane];
        }
        wave_lds_sync();
      }
    }
  }
  if (!merge) return;  // uniform across the workgroup
  __syncthreads();
  MergeWork<M>& MW = S.b.merge;
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) MW.tag[k * THREADS + t] = MERGE_EMPTY;
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) MW.cnt[k * THREADS + t] = 0u;
  for (int i = t; i < nt * (M / 4); i += THREADS) {
    const int r = i / (M / 4), c4 = i % (M / 4);
    const uint32_t l = perm[bbase + r].x;
    reinterpret_cast<float4*>(MW.g[r])[c4] = reinterpret_cast<const float4*>(gout + (size_t)l * M)[c4];
  }
  __syncthreads();
  // insert every pair's location; keep (entry, rank among the entry's pairs)
  uint32_t ent[MERGE_PPT];
  float wv[MERGE_PPT];
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) {
    const int pidx = k * THREADS + t;
    ent[k] = 0xFFFFFFFFu;
    wv[k] = 0.0f;
    if (pidx < nt * NB) {
      const int32_t loc = S.a.pairs.loc[pidx];
      wv[k] = S.a.pairs.w[pidx];
      if (loc >= 0) {
        uint32_t h = ((uint32_t)loc * 0x9E3779B1u) >> (32 - MERGE_HBITS);
        while (true) {
          const int32_t old = atomicCAS(&MW.tag[h], MERGE_EMPTY, loc);
          if (old == MERGE_EMPTY || old == loc) break;
          h = (h + 1) & (MERGE_H - 1);
        }
        const uint32_t sh = 16u * (h & 1u);
        const uint32_t rank = (atomicAdd(&MW.cnt[h >> 1], 1u << sh) >> sh) & 0xFFFFu;
        ent[k] = h | (rank << 16);
      }
    }
  }
  __syncthreads();
  // exclusive scan over the entries: group index and first position of each
  // occupied entry (this thread owns entries [t*HPT, (t+1)*HPT))
  uint32_t c[MERGE_HPT];
  uint32_t ng = 0, np = 0;
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) {
    const uint32_t wd = MW.cnt[t * (MERGE_HPT / 2) + k];
    c[2 * k] = wd & 0xFFFFu;
    c[2 * k + 1] = wd >> 16;
  }
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) {
    ng += c[k] ? 1u : 0u;
    np += c[k];
  }
  uint32_t sg = ng, sp = np;  // inclusive scan inside the wave
#pragma unroll
  for (int off = 1; off < WAVE; off <<= 1) {
    const uint32_t xg = __shfl_up(sg, off), xp = __shfl_up(sp, off);
    if (lane >= off) {
      sg += xg;
      sp += xp;
    }
  }
  if (lane == WAVE - 1) {
    MW.wsum[wave][0] = sg;
    MW.wsum[wave][1] = sp;
  }
  __syncthreads();
  uint32_t gb = sg - ng, pb = sp - np;
  for (int w = 0; w < wave; ++w) {
    gb += MW.wsum[w][0];
    pb += MW.wsum[w][1];
  }
  if (t == THREADS - 1) {
    MW.ngroups = gb + ng;
    S.a.grp.start[gb + ng] = (uint16_t)(pb + np);
  }
  uint32_t first[MERGE_HPT];
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) {
    first[k] = pb;
    if (c[k]) {
      S.a.grp.loc[gb] = MW.tag[t * MERGE_HPT + k];
      S.a.grp.start[gb] = (uint16_t)pb;
      ++gb;
      pb += c[k];
    }
  }
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) MW.cnt[t * (MERGE_HPT / 2) + k] = first[2 * k] | (first[2 * k + 1] << 16);
  __syncthreads();
  // pairs into group order (over the dead hash tags)
  float* pw = reinterpret_cast<float*>(MW.tag);
  uint8_t* pt = reinterpret_cast<uint8_t*>(MW.tag + MERGE_P);
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) {
    if (ent[k] != 0xFFFFFFFFu) {
      const uint32_t h = ent[k] & 0xFFFFu;
      const uint32_t pos = ((MW.cnt[h >> 1] >> (16u * (h & 1u))) & 0xFFFFu) + (ent[k] >> 16);
      pw[pos] = wv[k];
      pt[pos] = (uint8_t)((k * THREADS + t) / NB);
    }
  }
  __syncthreads();
  // one row per distinct location: M lanes (lane = column) sum w * G over its pairs
  constexpr int GROUPS = THREADS / M;
  const int col = t % M;
  const uint32_t ngroups = MW.ngroups;
  for (uint32_t gi = t / M; gi < ngroups; gi += GROUPS) {
    const uint32_t p0 = S.a.grp.start[gi], p1 = S.a.grp.start[gi + 1];
    float acc = 0.0f;
    for (uint32_t p = p0; p < p1; ++p) acc = fmaf(pw[p], MW.g[pt[p]][col], acc);
    unsafeAtomicAdd(gtab + (size_t)S.a.grp.loc[gi] * M + col, acc);
  }
}

// ---------------------------------------------------------------------------
// Access statistics (utilisation table): hist[s] += sum of the kernel weights
// of the pairs that read location s; then the fraction of locations read and
// the KL divergence of the weighted access distribution from uniform.

__global__ void __launch_bounds__(THREADS) k_access_hist(const float* __restrict__ q, Params P,
                                                         float* __restrict__ hist) {
  __shared__ SearchLds<WAVE> S;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  Search<NB> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<NB>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<false>(q, c.base, c.nl, P, FR, c.lane);
  for (int t = 0; t < c.nl; ++t) {
    const int count = srch.run(FR[t], read_sel(FR[t]), 0);
    if (c.lane < count) unsafeAtomicAdd(hist + W.nbr[0][c.lane].slot, W.wgt[0][c.lane]);
    wave_lds_sync();
  }
}

__global__ void k_fill_f64(double* __restrict__ p, int n, double v) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = v;
}

__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
  for (int mask = 1; mask < WAVE; mask <<= 1) x += __shfl_xor(x, mask);
  return x;
}

// acc[1] += sum h log h, acc[2] += sum h, acc[3] += #{h > 0} (fp64 partials per
// wave, one fp64 atomic per wave and sum).
__global__ void __launch_bounds__(THREADS) k_access_reduce(const float* __restrict__ hist, int64_t N,
                                                           double* __restrict__ acc) {
  double hl = 0.0, hs = 0.0, hc = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x; i < N; i += (int64_t)gridDim.x * THREADS) {
    const double h = hist[i];
    if (h > 0.0) {
      hl += h * log(h);
      hs += h;
      hc += 1.0;
    }
  }
  hl = wave_sum_f64(hl);
  hs = wave_sum_f64(hs);
  hc = wave_sum_f64(hc);
  if (threadIdx.x % WAVE == 0) {
    unsafeAtomicAdd(acc + 1, hl);
    unsafeAtomicAdd(acc + 2, hs);
    unsafeAtomicAdd(acc + 3, hc);
  }
}

// out[0] = used fraction, out[1] = KL(p || uniform) = log N + (sum h log h)/H - log H.
__global__ void k_access_finalize(double* __restrict__ out, int64_t N) {
  if (threadIdx.x != 0) return;
  const double H = out[2];
  out[0] = out[3] / (double)N;
  out[1] = H > 0.0 ? log((double)N) + out[1] / H - log(H) : 0.0;
}

// ---------------------------------------------------------------------------
// Adam step (Sec. 3.2: Adam on the memory parameters) on the rows of the table
// whose accumulated gradient row is not identically zero; the other rows keep
// value and moments.  M lanes per row (lane = column); the gradient row is
// cleared after use so the buffer is ready for the next accumulation.
struct AdamArgs {
  float lr, beta1, beta2, eps, om1, om2, bc1, bc2;  // om = 1 - beta, bc = 1 - beta^step (formed in fp64)
};

template <int DT, int M>
__global__ void __launch_bounds__(THREADS) k_sparse_adam(void* __restrict__ table, int64_t N,
                                                         float* __restrict__ grad, float* __restrict__ m1,
                                                         float* __restrict__ m2, AdamArgs a) {
  constexpr int RW = WAVE / M;  // rows per wave
  const int lane = threadIdx.x % WAVE;
  const int col = lane % M, sub = lane / M;
  const uint64_t seg = (M == WAVE) ? ~0ull : (((1ull << M) - 1ull) << (M * sub));
  const int64_t waves = (int64_t)gridDim.x * WAVES;
  for (int64_t rb = ((int64_t)blockIdx.x * WAVES + threadIdx.x / WAVE) * RW; rb < N; rb += waves * RW) {
    const int64_t r = rb + sub;
    const bool in = r < N;
    const size_t o = (size_t)(in ? r : 0) * M + col;
    const float g = in ? grad[o] : 0.0f;
    const bool touched = (__ballot(g != 0.0f) & seg) != 0;
    if (in && touched) {
      const float n1 = a.beta1 * m1[o] + a.om1 * g;
      const float n2 = a.beta2 * m2[o] + a.om2 * (g * g);
      m1[o] = n1;
      m2[o] = n2;
      const float step = a.lr * (n1 / a.bc1) / (sqrtf(n2 / a.bc2) + a.eps);
      if constexpr (DT == LRAM_F32) {
        float* t = reinterpret_cast<float*>(table) + o;
        *t = *t - step;
      } else {
        __bf16* t = reinterpret_cast<__bf16*>(table) + o;
        *t = (__bf16)((float)*t - step);
      }
      grad[o] = 0.0f;
    }
  }
}

// ---------------------------------------------------------------------------
// Host side.

thread_local int g_last_hip_error = 0;

int check_common(const float* q, int64_t B, int64_t H, const int32_t* K, int64_t* L, Params* P) {
  if (B < 0 || H < 0 || !K) return LRAM_EINVAL;
  if (H != 0 && B > INT64_MAX / H) return LRAM_EINVAL;
  *L = B * H;
  int64_t N = 1;
  for (int i = 0; i < 8; ++i) {
    if (K[i] < 2 || (K[i] & 1) || K[i] > KMAX) return LRAM_EBADK;
    N *= K[i];
    if (N >= (int64_t(1) << 31)) return LRAM_EBADK;
  }
  if (*L > 0) {
    if (!q || (reinterpret_cast<uintptr_t>(q) & 15)) return LRAM_EINVAL;
  }
  for (int i = 0; i < 8; ++i) {
    P->K[i] = K[i];
    P->twoK[i] = 2.0f * (float)K[i];
    uint32_t s = 1;
    for (int j = i + 1; j < 8; ++j) s *= (uint32_t)K[j];
    P->S[i] = s;
    P->cK[i] = (double)K[i] / (2.0 * 3.14159265358979323846);
  }
  P->N = (uint32_t)N;
  P->L = *L;
  // lookups per wave: up to 64, fewer for small batches so that every CU gets
  // work (about 16 waves per CU for 256 CUs)
  const int64_t target_waves = 256 * 16;
  int64_t lpw = (*L + target_waves - 1) / target_waves;
  P->lpw = (int32_t)(lpw < 1 ? 1 : (lpw > WAVE ? WAVE : lpw));
  return LRAM_OK;
}

int check_table(const void* table, int dtype, int64_t N, int32_t m, const Params& P, int64_t L) {
  if (dtype != LRAM_F32 && dtype != LRAM_BF16) return LRAM_EDTYPE;
  if (m != 32 && m != 64) return LRAM_EDTYPE;
  if (N != (int64_t)P.N) return LRAM_EBADK;
  if (L > 0 && (!table || (reinterpret_cast<uintptr_t>(table) & 15))) return LRAM_EINVAL;
  return LRAM_OK;
}

int launched() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    g_last_hip_error = (int)e;
    return LRAM_EHIP;
  }
  return LRAM_OK;
}

unsigned grid_for(const Params& P) {
  const int64_t per_block = (int64_t)P.lpw * WAVES;
  return (unsigned)((P.L + per_block - 1) / per_block);
}

template <template <int, int> class Launcher, typename... Args>
int dispatch(int dtype, int32_t m, Args... args) {
  if (dtype == LRAM_F32 && m == 32) return Launcher<LRAM_F32, 32>::go(args...);
  if (dtype == LRAM_F32 && m == 64) return Launcher<LRAM_F32, 64>::go(args...);
  if (dtype == LRAM_BF16 && m == 32) return Launcher<LRAM_BF16, 32>::go(args...);
  if (dtype == LRAM_BF16 && m == 64) return Launcher<LRAM_BF16, 64>::go(args...);
  return LRAM_EDTYPE;
}

template <int DT, int M>
struct FwdLaunch {
  static int go(const float* q, const Params& P, const void* table, void* out, bool th, hipStream_t s) {
    if (th)
      hipLaunchKernelGGL((k_forward<DT, M, true>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, out);
    else
      hipLaunchKernelGGL((k_forward<DT, M, false>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, out);
    return launched();
  }
};

// Workspace of the sorted scatter for n = 32 L pairs (each piece 256-byte aligned).
struct SortWs {
  uint32_t *k0, *k1, *hist, *totals;
  uint2 *v0, *v1;
  int64_t n;
  int nblocks;
  int64_t nh, nbt;
};

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

size_t sort_ws_layout(int64_t L, SortWs* ws, char* base) {
  const int64_t n = L * NB;
  const int nblocks = (int)((n + SORT_TILE - 1) / SORT_TILE);
  const int64_t nh = (int64_t)RADIX * nblocks;
  const int64_t nbt = (nh + SCAN_TILE - 1) / SCAN_TILE;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* ptr = base ? base + off : nullptr;
    off += align256(bytes);
    return ptr;
  };
  char* k0 = take(n * 4);
  char* k1 = take(n * 4);
  char* v0 = take(n * 8);
  char* v1 = take(n * 8);
  char* h = take(nh * 4);
  char* tt = take(nbt * 4);
  if (ws) {
    ws->k0 = (uint32_t*)k0; ws->k1 = (uint32_t*)k1; ws->v0 = (uint2*)v0; ws->v1 = (uint2*)v1;
    ws->hist = (uint32_t*)h; ws->totals = (uint32_t*)tt;
    ws->n = n; ws->nblocks = nblocks; ws->nh = nh; ws->nbt = nbt;
  }
  return off;
}

// Workspace of the batch-merged scatter for L lookups: the lookup sort (keys and
// (lookup, 0) values, double-buffered).
struct MergeWs {
  SortWs sort;
  uint32_t* shared;  // lookups sharing their closest lattice point (the merge gate)
};

size_t merge_ws_layout(int64_t L, MergeWs* ws, char* base) {
  const int64_t n = L;
  const int nblocks = (int)((n + SORT_TILE - 1) / SORT_TILE);
  const int64_t nh = (int64_t)RADIX * nblocks;
  const int64_t nbt = (nh + SCAN_TILE - 1) / SCAN_TILE;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* ptr = base ? base + off : nullptr;
    off += align256(bytes);
    return ptr;
  };
  char* k0 = take(n * 4);
  char* k1 = take(n * 4);
  char* v0 = take(n * 8);
  char* v1 = take(n * 8);
  char* h = take(nh * 4);
  char* tt = take(nbt * 4);
  char* sh = take(4);
  if (ws) {
    ws->shared = (uint32_t*)sh;
    SortWs& so = ws->sort;
    so.k0 = (uint32_t*)k0; so.k1 = (uint32_t*)k1; so.v0 = (uint2*)v0; so.v1 = (uint2*)v1;
    so.hist = (uint32_t*)h; so.totals = (uint32_t*)tt;
    so.n = n; so.nblocks = nblocks; so.nh = nh; so.nbt = nbt;
  }
  return off;
}

// Stable LSD radix sort of (key, value) pairs with keys in [0, N]; returns the
// buffers holding the result.
int radix_sort(const SortWs& ws, uint32_t N, hipStream_t s, uint32_t** kres, uint2** vres) {
  int bits = 0;
  while (bits < 32 && (N >> bits) != 0) ++bits;
  uint32_t* kin = ws.k0;
  uint32_t* kout = ws.k1;
  uint2* vin = ws.v0;
  uint2* vout = ws.v1;
  for (int shift = 0; shift < bits; shift += RADIX_BITS) {
    hipLaunchKernelGGL(k_radix_hist, dim3(ws.nblocks), dim3(THREADS), 0, s, kin, ws.n, shift, ws.hist, ws.nblocks);
    hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)ws.nbt), dim3(THREADS), 0, s, ws.hist, ws.nh, ws.totals);
    hipLaunchKernelGGL(k_scan_totals, dim3(1), dim3(THREADS), 0, s, ws.totals, ws.nbt);
    hipLaunchKernelGGL(k_scan_add, dim3((unsigned)ws.nbt), dim3(THREADS), 0, s, ws.hist, ws.nh, ws.totals);
    hipLaunchKernelGGL(k_radix_scatter, dim3(ws.nblocks), dim3(THREADS), 0, s, kin, vin, ws.n, shift, ws.hist,
                       ws.nblocks, kout, vout);
    if (int rc = launched()) return rc;
    std::swap(kin, kout);
    std::swap(vin, vout);
  }
  *kres = kin;
  *vres = vin;
  return LRAM_OK;
}

// q is the lookups' input: q [L][8], or z [L][16] when th (activation layer).
template <int DT, int M>
struct BwdAtomicLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq, bool th,
                hipStream_t s) {
    if (th)
      hipLaunchKernelGGL((k_backward<DT, M, false, true>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, (uint32_t*)nullptr, (uint2*)nullptr, (const uint32_t*)nullptr);
    else
      hipLaunchKernelGGL((k_backward<DT, M, false, false>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, (uint32_t*)nullptr, (uint2*)nullptr, (const uint32_t*)nullptr);
    return launched();
  }
};

template <int DT, int M>
struct BwdMergedLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const MergeWs& ws, bool th, hipStream_t s) {
    if (!gt) return BwdAtomicLaunch<DT, M>::go(q, P, table, g, gt, gq, th, s);
    const dim3 kgrid((unsigned)((P.L + THREADS - 1) / THREADS));
    if (th)
      hipLaunchKernelGGL(k_cell_key<true>, kgrid, dim3(THREADS), 0, s, q, P, ws.sort.k0, ws.sort.v0);
    else
      hipLaunchKernelGGL(k_cell_key<false>, kgrid, dim3(THREADS), 0, s, q, P, ws.sort.k0, ws.sort.v0);
    if (int rc = launched()) return rc;
    uint32_t* keys;
    uint2* perm;
    if (int rc = radix_sort(ws.sort, P.N, s, &keys, &perm)) return rc;
    // the gate: both scatters are launched, the count decides on the device
    // which one works (thinly spread queries have nothing to merge and keep
    // the atomic kernel's occupancy)
    hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(WAVE), 0, s, ws.shared, 0u);
    const int64_t cb = (P.L + THREADS - 1) / THREADS;
    hipLaunchKernelGGL(k_count_shared, dim3((unsigned)(cb < 2048 ? cb : 2048)), dim3(THREADS), 0, s,
                       (const uint32_t*)keys, P.L, ws.shared);
    if (th)
      hipLaunchKernelGGL((k_backward<DT, M, false, true>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, (uint32_t*)nullptr, (uint2*)nullptr, (const uint32_t*)ws.shared);
    else
      hipLaunchKernelGGL((k_backward<DT, M, false, false>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, (uint32_t*)nullptr, (uint2*)nullptr, (const uint32_t*)ws.shared);
    if (int rc = launched()) return rc;
    // one batch of at most MERGE_T lookups per workgroup
    Params Pm = P;
    Pm.lpw = P.lpw < MERGE_LPW ? P.lpw : MERGE_LPW;
    const int64_t per_block = (int64_t)Pm.lpw * WAVES;
    const dim3 grid((unsigned)((P.L + per_block - 1) / per_block));
    if (th)
      hipLaunchKernelGGL((k_backward_merged<DT, M, true>), grid, dim3(THREADS), 0, s, q, Pm, table, g, gt, gq,
                         (const uint32_t*)keys, (const uint2*)perm, (const uint32_t*)ws.shared);
    else
      hipLaunchKernelGGL((k_backward_merged<DT, M, false>), grid, dim3(THREADS), 0, s, q, Pm, table, g, gt, gq,
                         (const uint32_t*)keys, (const uint2*)perm, (const uint32_t*)ws.shared);
    return launched();
  }
};

template <int DT, int M>
struct BwdSortedLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const SortWs& ws, bool th, hipStream_t s) {
    if (th)
      hipLaunchKernelGGL((k_backward<DT, M, true, true>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, ws.k0, ws.v0, (const uint32_t*)nullptr);
    else
      hipLaunchKernelGGL((k_backward<DT, M, true, false>), dim3(grid_for(P)), dim3(THREADS), 0, s, q, P, table, g,
                         gt, gq, ws.k0, ws.v0, (const uint32_t*)nullptr);
    int rc = launched();
    if (rc || !gt) return rc;
    uint32_t* kin;
    uint2* vin;
    if ((rc = radix_sort(ws, P.N, s, &kin, &vin))) return rc;  // keys lie in [0, N]
    // span: 256 pairs per group, fewer when that would leave CUs idle (about
    // 32 groups per CU for 256 CUs)
    int64_t span = (ws.n + 256 * 32 - 1) / (256 * 32);
    span = span < SEG_BATCH ? SEG_BATCH : (span > SEG_SPAN ? SEG_SPAN : span);
    const int64_t groups = (ws.n + span - 1) / span;
    const int64_t per_block = THREADS / M;
    hipLaunchKernelGGL((k_segreduce<M>), dim3((unsigned)((groups + per_block - 1) / per_block)), dim3(THREADS), 0, s,
                       kin, vin, ws.n, P.N, g, gt, (int)span);
    return launched();
  }
};

// List width for k neighbours (k = LRAM_ALL: the whole support), 0 if k is not offered.
int list_width(int32_t k) {
  return k == LRAM_ALL ? KALL : ((k == 16 || k == 32 || k == 64) ? k : 0);
}

template <int DT, int M>
struct FwdKLaunch {
  static int go(const float* q, const Params& P, const void* table, void* out, int width, hipStream_t s) {
    const dim3 g(grid_for(P)), b(THREADS);
    switch (width) {
      case 16: hipLaunchKernelGGL((k_forward_k<DT, M, 16>), g, b, 0, s, q, P, table, out); break;
      case 64: hipLaunchKernelGGL((k_forward_k<DT, M, 64>), g, b, 0, s, q, P, table, out); break;
      case KALL: hipLaunchKernelGGL((k_forward_k<DT, M, KALL>), g, b, 0, s, q, P, table, out); break;
      default: hipLaunchKernelGGL((k_forward<DT, M, false>), g, b, 0, s, q, P, table, out); break;
    }
    return launched();
  }
};

template <int DT, int M>
struct BwdKLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq, int width,
                hipStream_t s) {
    const dim3 gr(grid_for(P)), b(THREADS);
    uint32_t* nk = nullptr;
    uint2* nv = nullptr;
    switch (width) {
      case 16: hipLaunchKernelGGL((k_backward<DT, M, false, false, 16>), gr, b, 0, s, q, P, table, g, gt, gq, nk, nv, nullptr); break;
      case 64: hipLaunchKernelGGL((k_backward<DT, M, false, false, 64>), gr, b, 0, s, q, P, table, g, gt, gq, nk, nv, nullptr); break;
      case KALL:
        hipLaunchKernelGGL((k_backward<DT, M, false, false, KALL>), gr, b, 0, s, q, P, table, g, gt, gq, nk, nv,
                           nullptr);
        break;
      default: hipLaunchKernelGGL((k_backward<DT, M, false, false, NB>), gr, b, 0, s, q, P, table, g, gt, gq, nk, nv, nullptr); break;
    }
    return launched();
  }
};

int forward_impl(const float* in, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype, int64_t N,
                 int32_t m, void* out, bool th, hipStream_t stream) {
  int64_t L;
  Params P;
  int rc = check_common(in, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!out || (reinterpret_cast<uintptr_t>(out) & 15)) return LRAM_EINVAL;
  return dispatch<FwdLaunch>(dtype, m, in, P, table, out, th, stream);
}

int resolve_mode(int64_t B, int64_t H, int mode, int* resolved);

int backward_impl(const float* in, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_in, int mode,
                  void* workspace, size_t ws_bytes, bool th, hipStream_t stream) {
  int64_t L;
  Params P;
  int rc = check_common(in, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if ((rc = resolve_mode(B, H, mode, &mode))) return rc;
  if (L == 0) return LRAM_OK;
  if (!grad_out || (reinterpret_cast<uintptr_t>(grad_out) & 15)) return LRAM_EINVAL;
  if (!grad_table && !grad_in) return LRAM_EINVAL;
  if (grad_table && (reinterpret_cast<uintptr_t>(grad_table) & 15)) return LRAM_EINVAL;
  if (grad_in && (reinterpret_cast<uintptr_t>(grad_in) & 15)) return LRAM_EINVAL;
  if (mode == LRAM_SCATTER_ATOMIC)
    return dispatch<BwdAtomicLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, th, stream);
  if (L > INT64_MAX / NB || L * NB >= (int64_t(1) << 32)) return LRAM_EINVAL;  // positions are 32-bit
  if (mode == LRAM_SCATTER_MERGED) {
    const size_t need = merge_ws_layout(L, nullptr, nullptr);
    if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LRAM_EWORKSPACE;
    MergeWs ws;
    merge_ws_layout(L, &ws, reinterpret_cast<char*>(workspace));
    return dispatch<BwdMergedLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, ws, th, stream);
  }
  const size_t need = sort_ws_layout(L, nullptr, nullptr);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LRAM_EWORKSPACE;
  SortWs ws;
  sort_ws_layout(L, &ws, reinterpret_cast<char*>(workspace));
  return dispatch<BwdSortedLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, ws, th, stream);
}

int resolve_mode(int64_t B, int64_t H, int mode, int* resolved) {
  if (!resolved || B < 0 || H < 0 || (H != 0 && B > INT64_MAX / H)) return LRAM_EINVAL;
  if (mode < LRAM_SCATTER_ATOMIC || mode > LRAM_SCATTER_AUTO) return LRAM_EMODE;
  *resolved = mode != LRAM_SCATTER_AUTO ? mode : (B * H >= AUTO_MERGE_MIN ? LRAM_SCATTER_MERGED : LRAM_SCATTER_ATOMIC);
  return LRAM_OK;
}

}  // namespace

extern "C" {

int lram_version(void) { return 100; }

const char* lram_strerror(int status) {
  switch (status) {
    case LRAM_OK: return "ok";
    case LRAM_EINVAL: return "invalid argument (null/misaligned pointer or negative size)";
    case LRAM_EBADK: return "invalid torus: every K_i must be even, 2 <= K_i <= 8192, N = prod K_i < 2^31";
    case LRAM_EDTYPE: return "unsupported table dtype or value dimension m";
    case LRAM_EWORKSPACE: return "workspace missing or too small";
    case LRAM_EMODE: return "unknown scatter mode";
    case LRAM_EHIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int lram_last_hip_error(void) { return g_last_hip_error; }

int lram_neighbors(const float* q, int64_t B, int64_t H, const int32_t K[8], int32_t* slot, float* w, float* d2,
                   void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!slot || !w) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_neighbors<NB>, dim3(grid_for(P)), dim3(THREADS), 0, (hipStream_t)stream, q, P, slot, w, d2);
  return launched();
}

int lram_forward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                 int64_t N, int32_t m, void* out, void* stream) {
  return forward_impl(q, B, H, K, table, dtype, N, m, out, false, (hipStream_t)stream);
}

int lram_theta_forward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                       int64_t N, int32_t m, void* out, void* stream) {
  return forward_impl(z, B, H, K, table, dtype, N, m, out, true, (hipStream_t)stream);
}

int lram_theta_coords(const float* z, int64_t B, int64_t H, const int32_t K[8], float* q, float* s, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(z, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!q || (reinterpret_cast<uintptr_t>(q) & 15)) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_theta_coords, dim3((unsigned)((L + THREADS - 1) / THREADS)), dim3(THREADS), 0,
                     (hipStream_t)stream, z, P, q, s);
  return launched();
}

int lram_scatter_mode_resolved(int64_t B, int64_t H, int mode, int* resolved) {
  return resolve_mode(B, H, mode, resolved);
}

int lram_backward_workspace_bytes(int64_t B, int64_t H, int32_t m, int mode, size_t* bytes) {
  if (!bytes || B < 0 || H < 0) return LRAM_EINVAL;
  if (m != 32 && m != 64) return LRAM_EDTYPE;
  if (int rc = resolve_mode(B, H, mode, &mode)) return rc;
  if (mode == LRAM_SCATTER_ATOMIC) {
    *bytes = 0;
    return LRAM_OK;
  }
  if (mode == LRAM_SCATTER_SORTED || mode == LRAM_SCATTER_MERGED) {
    if (H != 0 && B > INT64_MAX / H / NB) return LRAM_EINVAL;
    *bytes = mode == LRAM_SCATTER_SORTED ? sort_ws_layout(B * H, nullptr, nullptr)
                                         : merge_ws_layout(B * H, nullptr, nullptr);
    return LRAM_OK;
  }
  return LRAM_EMODE;
}

int lram_backward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, int mode,
                  void* workspace, size_t ws_bytes, void* stream) {
  return backward_impl(q, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_q, mode, workspace, ws_bytes,
                       false, (hipStream_t)stream);
}

int lram_theta_backward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                        int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_z, int mode,
                        void* workspace, size_t ws_bytes, void* stream) {
  return backward_impl(z, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_z, mode, workspace, ws_bytes,
                       true, (hipStream_t)stream);
}

int lram_access_histogram(const float* q, int64_t B, int64_t H, const int32_t K[8], float* hist, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!hist) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_access_hist, dim3(grid_for(P)), dim3(THREADS), 0, (hipStream_t)stream, q, P, hist);
  return launched();
}

int lram_access_stats(const float* hist, int64_t N, double* out, void* stream) {
  if (N <= 0 || !hist || !out || (reinterpret_cast<uintptr_t>(out) & 7)) return LRAM_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(k_fill_f64, dim3(1), dim3(WAVE), 0, s, out, 4, 0.0);
  const int64_t blocks = (N + THREADS - 1) / THREADS;
  hipLaunchKernelGGL(k_access_reduce, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(THREADS), 0, s, hist,
                     N, out);
  hipLaunchKernelGGL(k_access_finalize, dim3(1), dim3(WAVE), 0, s, out, N);
  return launched();
}

int lram_sparse_adam(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg, float* exp_avg_sq,
                     int64_t step, double lr, double beta1, double beta2, double eps, void* stream) {
  if (dtype != LRAM_F32 && dtype != LRAM_BF16) return LRAM_EDTYPE;
  if (m != 32 && m != 64) return LRAM_EDTYPE;
  if (N < 0 || step < 1 || !(lr >= 0.0) || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) ||
      !(eps >= 0.0))
    return LRAM_EINVAL;
  if (N == 0) return LRAM_OK;
  for (const void* ptr : {(const void*)table, (const void*)grad, (const void*)exp_avg, (const void*)exp_avg_sq})
    if (!ptr || (reinterpret_cast<uintptr_t>(ptr) & 15)) return LRAM_EINVAL;
  AdamArgs a;
  a.lr = (float)lr;
  a.beta1 = (float)beta1;
  a.beta2 = (float)beta2;
  a.eps = (float)eps;
  a.om1 = (float)(1.0 - beta1);
  a.om2 = (float)(1.0 - beta2);
  a.bc1 = (float)(1.0 - std::pow(beta1, (double)step));
  a.bc2 = (float)(1.0 - std::pow(beta2, (double)step));
  const int64_t rows_per_block = (int64_t)WAVES * (WAVE / m);
  int64_t blocks = (N + rows_per_block - 1) / rows_per_block;
  blocks = blocks < 16384 ? blocks : 16384;
  const dim3 g((unsigned)blocks), b(THREADS);
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LRAM_F32 && m == 32) hipLaunchKernelGGL((k_sparse_adam<LRAM_F32, 32>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, a);
  if (dtype == LRAM_F32 && m == 64) hipLaunchKernelGGL((k_sparse_adam<LRAM_F32, 64>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, a);
  if (dtype == LRAM_BF16 && m == 32) hipLaunchKernelGGL((k_sparse_adam<LRAM_BF16, 32>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, a);
  if (dtype == LRAM_BF16 && m == 64) hipLaunchKernelGGL((k_sparse_adam<LRAM_BF16, 64>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, a);
  return launched();
}

int lram_neighbors_k(const float* q, int64_t B, int64_t H, const int32_t K[8], int32_t k, int32_t* slot, float* w,
                     float* d2, void* stream) {
  const int width = list_width(k);
  if (!width) return LRAM_EINVAL;
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!slot || !w) return LRAM_EINVAL;
  const dim3 g(grid_for(P)), b(THREADS);
  hipStream_t s = (hipStream_t)stream;
  switch (width) {
    case 16: hipLaunchKernelGGL(k_neighbors<16>, g, b, 0, s, q, P, slot, w, d2); break;
    case 64: hipLaunchKernelGGL(k_neighbors<64>, g, b, 0, s, q, P, slot, w, d2); break;
    case KALL: hipLaunchKernelGGL(k_neighbors<KALL>, g, b, 0, s, q, P, slot, w, d2); break;
    default: hipLaunchKernelGGL(k_neighbors<NB>, g, b, 0, s, q, P, slot, w, d2); break;
  }
  return launched();
}

int lram_forward_k(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                   int64_t N, int32_t m, int32_t k, void* out, void* stream) {
  const int width = list_width(k);
  if (!width) return LRAM_EINVAL;
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!out || (reinterpret_cast<uintptr_t>(out) & 15)) return LRAM_EINVAL;
  return dispatch<FwdKLaunch>(dtype, m, q, P, table, out, width, (hipStream_t)stream);
}

int lram_backward_k(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                    int64_t N, int32_t m, int32_t k, const float* grad_out, float* grad_table, float* grad_q,
                    void* stream) {
  const int width = list_width(k);
  if (!width) return LRAM_EINVAL;
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!grad_out || (reinterpret_cast<uintptr_t>(grad_out) & 15)) return LRAM_EINVAL;
  if (!grad_table && !grad_q) return LRAM_EINVAL;
  if (grad_table && (reinterpret_cast<uintptr_t>(grad_table) & 15)) return LRAM_EINVAL;
  if (grad_q && (reinterpret_cast<uintptr_t>(grad_q) & 15)) return LRAM_EINVAL;
  return dispatch<BwdKLaunch>(dtype, m, q, P, table, grad_out, grad_table, grad_q, width, (hipStream_t)stream);
}

}  // extern "C"
