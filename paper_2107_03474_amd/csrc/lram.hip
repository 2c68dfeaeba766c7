// liblram -- LRAM lattice lookup for AMD Instinct MI355X (gfx950, CDNA4).
//
// Goucher & Troll, "Differentiable Random Access Memory using Lattices":
// lookup phi (Sec. 2.2) over the lattice Lambda = 2*E8 (Sec. 2.4) with the
// kernel f(r) = (1 - r^2/8)^4 (Sec. 2.5), truncated to the 32 closest points
// and found through the symmetry reduction of Sec. 2.6, plus its backward.
//
// Work decomposition (one wave = 64 lanes):
//   phase A  lane-per-lookup: wrap, E8 closest point (D8 and D8+1/2 decoders
//            with a parity fix), and the signed permutation that carries the
//            offset into the fundamental region F; the result (a "frame") goes
//            to LDS, 64 lookups per wave.
//   phase B  wave-per-lookup: the wave builds three 8x8 per-query tables in LDS
//            (squared coordinate error, location contribution, coordinate
//            error) indexed by (original coordinate, candidate coordinate
//            value), scans the 232 candidate points of F (4 per lane) with one
//            v_perm + one LDS read per coordinate, selects the closest 32 with
//            ballot/popcount bisection on the fp32 distance bits, and then
//            gather-reduces (forward) or scatters and forms dq (backward) with
//            coalesced 16-byte row reads.
// No MFMA: the path is a gather / scatter bound by HBM, not a contraction.

#include <hip/hip_runtime.h>
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

// ties at the 32nd distance involve points of the support (at most 121 of them)
constexpr int TIE_MAX = 128;
constexpr uint32_t KEY_INF = 0x7F800000u;   // +inf: never selected
constexpr uint32_t KEY_8 = 0x41000000u;     // 8.0f: support boundary (open ball)
constexpr uint32_t KEY_4 = 0x40800000u;     // 4.0f: fewer than 32 points are ever closer
constexpr uint32_t KEY_SUSPECT = 0x40FFF7CFu;  // 7.999f

__constant__ signed char c_strict[E8_NSTRICT][8] = E8_STRICT_INIT;
__constant__ signed char c_boundary[E8_NBOUNDARY][8] = E8_BOUNDARY_INIT;

struct Params {
  int32_t K[8];
  uint32_t S[8];     // mixed-radix strides of the location map, S_7 = 1
  float twoK[8];     // torus side at the Lambda scale
  uint32_t N;
  int64_t L;
};

// Per-lookup frame written by phase A (112 bytes, 16-byte aligned fields).
struct alignas(16) Frame {
  float x[8];         // Lambda-scale query, wrapped
  int32_t c[8];       // closest lattice point
  uint32_t sel[8];    // v_perm selector for original coordinate i: byte r_i of the candidate
  uint32_t misc;      // bits 0-7: sign flips s'_i = -1; bit 8: query finite
  uint32_t pad[3];
};

// A selected neighbour as handed from the search to the gather / scatter.
struct alignas(16) Nbr {
  uint32_t lo, hi;    // packed candidate bytes (F coordinates)
  uint32_t dbits;     // fp32 recipe distance^2 bits
  int32_t slot;       // location, -1 for padding
};

struct alignas(16) WaveLds {
  Frame frames[WAVE];
  Nbr nbr[NB];
  float wgt[NB];
  uint32_t tie[TIE_MAX][2];
};

struct alignas(16) BlockLds {
  // per-query tables, [coordinate i][wave w][value v] -> byte i*256 + w*64 + 4v
  float qt[8 * 64];
  uint32_t st[8 * 64];
  float et[8 * 64];
  WaveLds wave[WAVES];
};

__device__ __forceinline__ float lds_f32(const float* base, uint32_t byte_off) {
  return *reinterpret_cast<const float*>(reinterpret_cast<const char*>(base) + byte_off);
}
__device__ __forceinline__ uint32_t lds_u32(const uint32_t* base, uint32_t byte_off) {
  return *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(base) + byte_off);
}

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0)); }

__device__ __forceinline__ int prefix_count(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

// Orders LDS traffic between lanes of one wave: the wave's LDS operations
// execute in issue order, so a compiler barrier plus waiting for the
// outstanding LDS operations is enough.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;  // quiet NaN
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
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

__device__ void make_frame(const float* __restrict__ q, bool have, const Params& P, Frame& F) {
  float x[8];
  bool valid = have;
  if (have) {
    float4 a = reinterpret_cast<const float4*>(q)[0];
    float4 b = reinterpret_cast<const float4*>(q)[1];
    float qq[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
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
  int c[8];
  float a[8];
  uint32_t neg = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    c[i] = odd ? 2 * r1[i] + 1 : 2 * r0[i];
    float y = x[i] - (float)c[i];
    a[i] = fabsf(y);
    neg |= (y < 0.0f ? 1u : 0u) << i;
  }
  // rank of |y_i| in descending order (ties by index): F position of coordinate i
  int r[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int ri = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (j != i) ri += (a[j] > a[i] || (a[j] == a[i] && j < i)) ? 1 : 0;
    r[i] = ri;
  }
  // only even numbers of sign changes are isometries of Lambda: fix the parity
  // on the coordinate that lands last (smallest |y|)
  if (__popc(neg) & 1) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (r[i] == 7) neg ^= 1u << i;
  }
  float4* fx = reinterpret_cast<float4*>(F.x);
  fx[0] = make_float4(x[0], x[1], x[2], x[3]);
  fx[1] = make_float4(x[4], x[5], x[6], x[7]);
  int4* fc = reinterpret_cast<int4*>(F.c);
  fc[0] = make_int4(c[0], c[1], c[2], c[3]);
  fc[1] = make_int4(c[4], c[5], c[6], c[7]);
  uint4* fs = reinterpret_cast<uint4*>(F.sel);
  fs[0] = make_uint4(0x0C0C0C00u | r[0], 0x0C0C0C00u | r[1], 0x0C0C0C00u | r[2], 0x0C0C0C00u | r[3]);
  fs[1] = make_uint4(0x0C0C0C00u | r[4], 0x0C0C0C00u | r[5], 0x0C0C0C00u | r[6], 0x0C0C0C00u | r[7]);
  F.misc = neg | (valid ? 0x100u : 0u);
}

// ---------------------------------------------------------------------------
// Phase B helpers.

// Packed candidate bytes for lane-slot idx of a list: byte j = 4*(p_j - CMIN) + 64*w.
__device__ __forceinline__ void pack_candidate(const signed char (&p)[8], uint32_t wbyte, uint32_t& lo,
                                               uint32_t& hi) {
  lo = hi = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    lo |= ((uint32_t)(4 * (p[j] - CMIN)) + wbyte) << (8 * j);
    hi |= ((uint32_t)(4 * (p[j + 4] - CMIN)) + wbyte) << (8 * j);
  }
}

template <int LIST>
__device__ __forceinline__ bool load_candidate(int idx, uint32_t wbyte, uint32_t& lo, uint32_t& hi) {
  constexpr int n = LIST == 0 ? E8_NSTRICT : E8_NBOUNDARY;
  if (idx >= n) {
    lo = hi = 0;
    return false;
  }
  signed char p[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) p[j] = LIST == 0 ? c_strict[idx][j] : c_boundary[idx][j];
  pack_candidate(p, wbyte, lo, hi);
  return true;
}

// Recipe distance^2 of candidate (lo,hi): sum over original coordinates i, in
// order, of the per-query table entry (x_i - k_i)^2 (already fp32-rounded).
__device__ __forceinline__ float cand_d2(const float* qt, uint32_t lo, uint32_t hi, const uint32_t (&sel)[8]) {
  float d = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t a = __builtin_amdgcn_perm(hi, lo, sel[i]);
    float v = lds_f32(qt, a + 256u * i);
    d = (i == 0) ? v : d + v;
  }
  return d;
}

__device__ __forceinline__ int32_t cand_slot(const uint32_t* st, uint32_t lo, uint32_t hi,
                                             const uint32_t (&sel)[8]) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) m += lds_u32(st, __builtin_amdgcn_perm(hi, lo, sel[i]) + 256u * i);
  return (int32_t)(m >> 1);
}

// Lexicographic key of the lattice point itself (only consulted between equal
// (distance, location) pairs, which requires a torus side of 2).
__device__ __forceinline__ uint32_t cand_liftkey(uint32_t lo, uint32_t hi, const uint32_t (&sel)[8],
                                                 const Frame& F) {
  uint32_t key = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t a = __builtin_amdgcn_perm(hi, lo, sel[i]);
    int p = (int)((a & 63u) >> 2) + CMIN;
    int k = ((F.misc >> i) & 1u) ? F.c[i] - p : F.c[i] + p;
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

// Selection of the closest 32 (Sec. 2.6) over NS candidate slots per lane.
// Result: pick bit s set for each selected slot of this lane; returns the
// number selected; *suspect is set when a point of the boundary list could
// enter the selection (the 32nd distance is within 1e-3 of the support edge,
// or fewer than 32 points are in the support).
template <int NS>
__device__ int select32(const uint32_t (&key)[NS], const uint32_t (&lo)[NS], const uint32_t (&hi)[NS],
                        const uint32_t (&sel)[8], const Frame& F, const uint32_t* st, WaveLds& W,
                        uint32_t& pick, bool& suspect) {
  const int lane = lane_id();
  pick = 0;
  const int n8 = count_below(key, KEY_8);
  if (n8 <= NB) {
#pragma unroll
    for (int s = 0; s < NS; ++s) pick |= (key[s] < KEY_8 ? 1u : 0u) << s;
    suspect = true;
    return n8;
  }
  // bisection on the (monotone) bit patterns of non-negative floats:
  // invariant count(< lo) < 32 < count(< hi)
  uint32_t lo_k = KEY_4, hi_k = KEY_8;
  int c = count_below(key, lo_k);
  if (c == NB) {
#pragma unroll
    for (int s = 0; s < NS; ++s) pick |= (key[s] < lo_k ? 1u : 0u) << s;
    suspect = false;
    return NB;
  }
  if (c > NB) {
    hi_k = lo_k;
    lo_k = 0;
  }
  while (hi_k - lo_k > 1) {
    uint32_t mid = lo_k + ((hi_k - lo_k) >> 1);
    c = count_below(key, mid);
    if (c == NB) {
#pragma unroll
      for (int s = 0; s < NS; ++s) pick |= (key[s] < mid ? 1u : 0u) << s;
      suspect = mid > KEY_SUSPECT;
      return NB;
    }
    if (c < NB)
      lo_k = mid;
    else
      hi_k = mid;
  }
  // Several candidates share the distance bits lo_k at the 32nd place: take
  // the ones below, then the tied ones in (location, lattice point) order.
  const int below = count_below(key, lo_k);
  const int need = NB - below;
  suspect = lo_k > KEY_SUSPECT;
  int nt = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const bool tied = key[s] == lo_k;
    const uint64_t m = __ballot(tied);
    const int pos = nt + prefix_count(m);
    if (tied && pos < TIE_MAX) {
      W.tie[pos][0] = (uint32_t)cand_slot(st, lo[s], hi[s], sel);
      W.tie[pos][1] = cand_liftkey(lo[s], hi[s], sel, F);
    }
    nt += __popcll(m);
  }
  wave_lds_sync();
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    pick |= (key[s] < lo_k ? 1u : 0u) << s;
    if (key[s] == lo_k) {
      const uint32_t ms = (uint32_t)cand_slot(st, lo[s], hi[s], sel);
      const uint32_t mk = cand_liftkey(lo[s], hi[s], sel, F);
      int rank = 0;
      const int ntc = nt < TIE_MAX ? nt : TIE_MAX;
      for (int e = 0; e < ntc; ++e) {
        const uint32_t es = W.tie[e][0], ek = W.tie[e][1];
        rank += (es < ms || (es == ms && ek < mk)) ? 1 : 0;
      }
      if (rank < need) pick |= 1u << s;
    }
  }
  (void)lane;
  wave_lds_sync();
  return NB;
}

// Writes the picked slots into W.nbr[0..count) (order: slot-major, then lane).
template <int NS>
__device__ __forceinline__ void compact(const uint32_t pick, const uint32_t (&key)[NS], const uint32_t (&lo)[NS],
                                        const uint32_t (&hi)[NS], WaveLds& W) {
  int base = 0;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const bool p = (pick >> s) & 1u;
    const uint64_t m = __ballot(p);
    if (p) {
      Nbr& n = W.nbr[base + prefix_count(m)];
      n.lo = lo[s];
      n.hi = hi[s];
      n.dbits = key[s];
    }
    base += __popcll(m);
  }
}

struct Search {
  const Params& P;
  BlockLds& S;
  WaveLds& W;
  int wave;
  int lane;
  uint32_t wbyte;
  uint32_t lo[NS_STRICT], hi[NS_STRICT];
  bool ok[NS_STRICT];
  // lane constants of the table build: coordinate i = lane/8, value v = lane%8
  int ti, tv, tK;
  uint32_t tS;
  uint32_t toff;  // byte offset of entry (i, w, v)

  __device__ Search(const Params& p, BlockLds& s, int w, int l)
      : P(p), S(s), W(s.wave[w]), wave(w), lane(l), wbyte(64u * (uint32_t)w) {
#pragma unroll
    for (int k = 0; k < NS_STRICT; ++k) ok[k] = load_candidate<0>(lane + WAVE * k, wbyte, lo[k], hi[k]);
    ti = lane >> 3;
    tv = lane & 7;
    tK = 0;
    tS = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i == ti) {
        tK = P.K[i];
        tS = P.S[i];
      }
    toff = 256u * ti + wbyte + 4u * tv;
  }

  // Per-query tables for frame F: entry (i, v) describes the lattice
  // coordinate k_i = c_i + s'_i (v + CMIN).
  __device__ void build_tables(const Frame& F) {
    const float xi = F.x[ti];
    const int ci = F.c[ti];
    const int p = tv + CMIN;
    const int k = ((F.misc >> ti) & 1u) ? ci - p : ci + p;
    const float e = xi - (float)k;
    const float e2 = e * e;
    const int par = k & 1;
    int Y = (k - par) >> 1;
    // Y is within one period of [0, K) either side plus 3
    while (Y < 0) Y += tK;
    while (Y >= tK) Y -= tK;
    const uint32_t sl = (uint32_t)Y * tS + ((ti == 0 && par) ? P.N : 0u);
    *reinterpret_cast<float*>(reinterpret_cast<char*>(S.qt) + toff) = e2;
    *reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(S.st) + toff) = sl;
    *reinterpret_cast<float*>(reinterpret_cast<char*>(S.et) + toff) = e;
  }

  // Full neighbour search for frame F.  Leaves W.nbr[0..32) with
  // (lo, hi, dbits, slot) and W.wgt with the fp32 recipe weights, padded with
  // slot -1 / weight 0; returns the number of real neighbours.
  __device__ int run(const Frame& F, uint32_t (&sel)[8]) {
    const uint4* fs = reinterpret_cast<const uint4*>(F.sel);
    const uint4 s0 = fs[0], s1 = fs[1];
    sel[0] = s0.x; sel[1] = s0.y; sel[2] = s0.z; sel[3] = s0.w;
    sel[4] = s1.x; sel[5] = s1.y; sel[6] = s1.z; sel[7] = s1.w;
    int count = 0;
    if (F.misc & 0x100u) {
      build_tables(F);
      wave_lds_sync();
      uint32_t key[NS_STRICT];
#pragma unroll
      for (int k = 0; k < NS_STRICT; ++k)
        key[k] = ok[k] ? __float_as_uint(cand_d2(S.qt, lo[k], hi[k], sel)) : KEY_INF;
      uint32_t pick;
      bool suspect;
      count = select32<NS_STRICT>(key, lo, hi, sel, F, S.st, W, pick, suspect);
      if (!suspect) {
        compact<NS_STRICT>(pick, key, lo, hi, W);
      } else {
        // rare: rescan together with the points at distance exactly sqrt(8) from F
        uint32_t key7[NS_ALL], lo7[NS_ALL], hi7[NS_ALL];
#pragma unroll
        for (int k = 0; k < NS_STRICT; ++k) {
          key7[k] = key[k];
          lo7[k] = lo[k];
          hi7[k] = hi[k];
        }
#pragma unroll
        for (int k = 0; k < NS_BOUND; ++k) {
          const bool okb = load_candidate<1>(lane + WAVE * k, wbyte, lo7[NS_STRICT + k], hi7[NS_STRICT + k]);
          key7[NS_STRICT + k] =
              okb ? __float_as_uint(cand_d2(S.qt, lo7[NS_STRICT + k], hi7[NS_STRICT + k], sel)) : KEY_INF;
        }
        bool suspect7;
        count = select32<NS_ALL>(key7, lo7, hi7, sel, F, S.st, W, pick, suspect7);
        compact<NS_ALL>(pick, key7, lo7, hi7, W);
      }
      wave_lds_sync();
    }
    // locations and weights, one neighbour per lane
    if (lane < NB) {
      Nbr& n = W.nbr[lane];
      if (lane < count) {
        n.slot = cand_slot(S.st, n.lo, n.hi, sel);
        const float d = __uint_as_float(n.dbits);
        const float u = 1.0f - d * 0.125f;
        const float u2 = u * u;
        W.wgt[lane] = u2 * u2;
      } else {
        n.lo = n.hi = 0;
        n.dbits = KEY_INF;
        n.slot = -1;
        W.wgt[lane] = 0.0f;
      }
    }
    wave_lds_sync();
    return count;
  }
};

// Phase A for the wave's 64 lookups starting at `base`.
__device__ __forceinline__ void phase_a(const float* __restrict__ q, int64_t base, const Params& P, WaveLds& W,
                                        int lane) {
  const int64_t l = base + lane;
  const bool have = l < P.L;
  make_frame(q + (have ? l : 0) * 8, have, P, W.frames[lane]);
  wave_lds_sync();
}

// ---------------------------------------------------------------------------
// Kernels.

__global__ void __launch_bounds__(THREADS) k_neighbors(const float* __restrict__ q, Params P,
                                                       int32_t* __restrict__ slot_out, float* __restrict__ w_out,
                                                       float* __restrict__ d2_out) {
  __shared__ BlockLds S;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int64_t base = ((int64_t)blockIdx.x * WAVES + wave) * WAVE;
  if (base >= P.L) return;
  Search srch(P, S, wave, lane);
  WaveLds& W = S.wave[wave];
  phase_a(q, base, P, W, lane);
  const int nl = (int)min<int64_t>(WAVE, P.L - base);
  for (int t = 0; t < nl; ++t) {
    uint32_t sel[8];
    const Frame& F = W.frames[t];
    const int count = srch.run(F, sel);
    const int64_t l = base + t;
    if (lane < NB) {
      // order the list by (distance bits, location, lattice point)
      const Nbr me = W.nbr[lane];
      int rank = lane;
      if (lane < count) {
        const uint32_t mk = cand_liftkey(me.lo, me.hi, sel, F);
        rank = 0;
        for (int e = 0; e < count; ++e) {
          const Nbr o = W.nbr[e];
          bool less = o.dbits < me.dbits || (o.dbits == me.dbits && o.slot < me.slot);
          if (o.dbits == me.dbits && o.slot == me.slot && e != lane) less = cand_liftkey(o.lo, o.hi, sel, F) < mk;
          rank += less ? 1 : 0;
        }
      }
      slot_out[l * NB + rank] = me.slot;
      w_out[l * NB + rank] = W.wgt[lane];
      if (d2_out) d2_out[l * NB + rank] = __uint_as_float(me.dbits);
    }
    wave_lds_sync();
  }
}

template <int DT, int M>
struct RowGeom {
  static constexpr int ES = DT == LRAM_F32 ? 4 : 2;      // table element bytes
  static constexpr int RB = M * ES;                       // row bytes
  static constexpr int LPR = RB / 16;                     // lanes per row (16 B each)
  static constexpr int RPP = WAVE / LPR;                  // rows per pass
  static constexpr int NP = NB / RPP;                     // passes
  static constexpr int EPC = 16 / ES;                     // elements per 16-byte chunk
  static_assert(RB % 16 == 0 && LPR <= WAVE && NB % RPP == 0, "row geometry");
};

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

template <int DT, int M>
__global__ void __launch_bounds__(THREADS) k_forward(const float* __restrict__ q, Params P,
                                                     const void* __restrict__ table, void* __restrict__ out) {
  using G = RowGeom<DT, M>;
  __shared__ BlockLds S;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int64_t base = ((int64_t)blockIdx.x * WAVES + wave) * WAVE;
  if (base >= P.L) return;
  Search srch(P, S, wave, lane);
  WaveLds& W = S.wave[wave];
  phase_a(q, base, P, W, lane);
  const int nl = (int)min<int64_t>(WAVE, P.L - base);
  const int rsub = lane / G::LPR, ch = lane % G::LPR;
  const char* tb = reinterpret_cast<const char*>(table);
  for (int t = 0; t < nl; ++t) {
    uint32_t sel[8];
    srch.run(W.frames[t], sel);
    uint4 v[G::NP];
    float w[G::NP];
#pragma unroll
    for (int p = 0; p < G::NP; ++p) {
      const int j = p * G::RPP + rsub;
      const int32_t s = W.nbr[j].slot;
      w[p] = W.wgt[j];
      v[p] = s >= 0 ? *reinterpret_cast<const uint4*>(tb + (size_t)s * G::RB + ch * 16) : make_uint4(0, 0, 0, 0);
    }
    float acc[G::EPC];
#pragma unroll
    for (int e = 0; e < G::EPC; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int p = 0; p < G::NP; ++p) {
      float f[G::EPC];
      unpack16<DT, G::EPC>(v[p], f);
#pragma unroll
      for (int e = 0; e < G::EPC; ++e) acc[e] = fmaf(w[p], f[e], acc[e]);
    }
#pragma unroll
    for (int mask = G::LPR; mask < WAVE; mask <<= 1)
#pragma unroll
      for (int e = 0; e < G::EPC; ++e) acc[e] += __shfl_xor(acc[e], mask);
    if (rsub == 0) {
      const int64_t l = base + t;
      char* ob = reinterpret_cast<char*>(out) + (size_t)l * G::RB + ch * 16;
      if constexpr (DT == LRAM_F32) {
        *reinterpret_cast<float4*>(ob) = make_float4(acc[0], acc[1], acc[2], acc[3]);
      } else {
        uint4 o;
        o.x = f32_to_bf16_rne(acc[0]) | (f32_to_bf16_rne(acc[1]) << 16);
        o.y = f32_to_bf16_rne(acc[2]) | (f32_to_bf16_rne(acc[3]) << 16);
        o.z = f32_to_bf16_rne(acc[4]) | (f32_to_bf16_rne(acc[5]) << 16);
        o.w = f32_to_bf16_rne(acc[6]) | (f32_to_bf16_rne(acc[7]) << 16);
        *reinterpret_cast<uint4*>(ob) = o;
      }
    }
    wave_lds_sync();
  }
}

// Backward, fused with the query gradient: per lookup, read the 32 rows once
// for <G, v_j> and form dq from the coordinate errors.  The value gradient is
// either added straight into grad_table with fp32 atomics (EMIT = false), or
// emitted as (location, (lookup, w_j)) pairs for the sorted segmented
// reduction (EMIT = true; padding gets the key N, which sorts last).
template <int DT, int M, bool EMIT>
__global__ void __launch_bounds__(THREADS) k_backward(const float* __restrict__ q, Params P,
                                                      const void* __restrict__ table,
                                                      const float* __restrict__ gout, float* __restrict__ gtab,
                                                      float* __restrict__ gq, uint32_t* __restrict__ pair_key,
                                                      uint2* __restrict__ pair_val) {
  using G = RowGeom<DT, M>;
  constexpr int ICOORD = G::LPR >= 8 ? 1 : 8 / G::LPR;  // query coordinates per lane
  __shared__ BlockLds S;
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int64_t base = ((int64_t)blockIdx.x * WAVES + wave) * WAVE;
  if (base >= P.L) return;
  Search srch(P, S, wave, lane);
  WaveLds& W = S.wave[wave];
  phase_a(q, base, P, W, lane);
  const int nl = (int)min<int64_t>(WAVE, P.L - base);
  const int rsub = lane / G::LPR, ch = lane % G::LPR;
  const char* tb = reinterpret_cast<const char*>(table);
  for (int t = 0; t < nl; ++t) {
    uint32_t sel[8];
    const Frame& F = W.frames[t];
    const int count = srch.run(F, sel);
    const int64_t l = base + t;
    float dq[ICOORD];
#pragma unroll
    for (int c = 0; c < ICOORD; ++c) dq[c] = 0.0f;
    if (count > 0) {
      float g[G::EPC];
      const float* gp = gout + (size_t)l * M + ch * G::EPC;
#pragma unroll
      for (int e = 0; e < G::EPC; e += 4) {
        const float4 gv = *reinterpret_cast<const float4*>(gp + e);
        g[e] = gv.x; g[e + 1] = gv.y; g[e + 2] = gv.z; g[e + 3] = gv.w;
      }
      // value-gradient scatter: M consecutive lanes own one gradient row, so each
      // atomic instruction covers 64/M whole rows (full-line requests at L2)
      if (!EMIT && gtab) {
        constexpr int RA = WAVE / M;
        const int col = lane % M;
        const float gc = gout[(size_t)l * M + col];
#pragma unroll 4
        for (int k = 0; k < NB / RA; ++k) {
          const int j = k * RA + lane / M;
          const int32_t s = W.nbr[j].slot;
          if (s >= 0) unsafeAtomicAdd(gtab + (size_t)s * M + col, W.wgt[j] * gc);
        }
      }
      uint4 v[G::NP];
      int32_t sl[G::NP];
#pragma unroll
      for (int p = 0; p < G::NP; ++p) {
        const int j = p * G::RPP + rsub;
        sl[p] = W.nbr[j].slot;
        v[p] = sl[p] >= 0 ? *reinterpret_cast<const uint4*>(tb + (size_t)sl[p] * G::RB + ch * 16)
                          : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int p = 0; p < G::NP; ++p) {
        const int j = p * G::RPP + rsub;
        float f[G::EPC];
        unpack16<DT, G::EPC>(v[p], f);
        float pd = 0.0f;
#pragma unroll
        for (int e = 0; e < G::EPC; ++e) pd = fmaf(g[e], f[e], pd);
        // <G, v_j>: sum over the LPR lanes of this row
#pragma unroll
        for (int mask = 1; mask < G::LPR; mask <<= 1) pd += __shfl_xor(pd, mask);
        if (gq && sl[p] >= 0) {
          const Nbr n = W.nbr[j];
          const float u = 1.0f - __uint_as_float(n.dbits) * 0.125f;
          const float a = -2.0f * u * u * u * pd;
#pragma unroll
          for (int c = 0; c < ICOORD; ++c) {
            const int i = ch + c * G::LPR;
            if (i < 8) {
              const uint32_t ab = __builtin_amdgcn_perm(n.hi, n.lo, F.sel[i]);
              dq[c] = fmaf(a, lds_f32(S.et, ab + 256u * i), dq[c]);
            }
          }
        }
      }
    }
    if (EMIT && gtab && lane < NB) {
      const int32_t sl = W.nbr[lane].slot;
      pair_key[l * NB + lane] = sl >= 0 ? (uint32_t)sl : P.N;
      pair_val[l * NB + lane] = make_uint2((uint32_t)l, __float_as_uint(W.wgt[lane]));
    }
    if (gq) {
#pragma unroll
      for (int mask = G::LPR; mask < WAVE; mask <<= 1)
#pragma unroll
        for (int c = 0; c < ICOORD; ++c) dq[c] += __shfl_xor(dq[c], mask);
      if (rsub == 0) {
#pragma unroll
        for (int c = 0; c < ICOORD; ++c) {
          const int i = ch + c * G::LPR;
          if (i < 8) gq[l * 8 + i] = dq[c];
        }
      }
    }
    wave_lds_sync();
  }
}


// ---------------------------------------------------------------------------
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
__global__ void __launch_bounds__(THREADS) k_radix_scatter(const uint32_t* __restrict__ kin,
                                                           const uint2* __restrict__ vin, int64_t n, int shift,
                                                           const uint32_t* __restrict__ offs, int nblocks,
                                                           uint32_t* __restrict__ kout, uint2* __restrict__ vout) {
  __shared__ uint32_t run_cnt[RADIX];
  __shared__ uint32_t wave_cnt[WAVES][RADIX];
  __shared__ uint32_t base_off[RADIX];
  const int t = threadIdx.x, w = t / WAVE, lane = t % WAVE;
  run_cnt[t] = 0;
  base_off[t] = offs[(int64_t)t * nblocks + blockIdx.x];
#pragma unroll
  for (int k = 0; k < WAVES; ++k) wave_cnt[k][t] = 0;
  __syncthreads();
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (WAVE - lane));
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE;
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int64_t i = base + r * THREADS + t;
    const bool valid = i < n;
    const uint32_t key = valid ? kin[i] : 0u;
    const uint2 val = valid ? vin[i] : make_uint2(0, 0);
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
        const uint32_t c = wave_cnt[k][t];
        wave_cnt[k][t] = run;
        run += c;
      }
      run_cnt[t] = run;
    }
    __syncthreads();
    if (valid) {
      const uint32_t pos = base_off[d] + wave_cnt[w][d] + (uint32_t)rank;
      kout[pos] = key;
      vout[pos] = val;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < WAVES; ++k) wave_cnt[k][t] = 0;
    __syncthreads();
  }
}

// Segmented reduction of the sorted pairs: one wave per 64 consecutive pairs
// (lane = pair).  Each lane forms w * G[lookup] in column groups of 16, a
// segmented inclusive scan over the lanes sums every run of equal locations,
// and the last lane of each run writes the row: a plain read-modify-write when
// the whole run lies inside these 64 pairs (no other wave touches that row),
// fp32 atomics for the runs cut by the chunk edges.
template <int M>
__global__ void __launch_bounds__(THREADS) k_segreduce(const uint32_t* __restrict__ keys,
                                                       const uint2* __restrict__ vals, int64_t n, uint32_t N,
                                                       const float* __restrict__ gout, float* __restrict__ gtab) {
  const int lane = threadIdx.x % WAVE;
  const int64_t chunk = (int64_t)blockIdx.x * WAVES + threadIdx.x / WAVE;
  const int64_t p = chunk * WAVE + lane;
  if (chunk * WAVE >= n) return;
  const bool valid = p < n;
  const uint32_t key = valid ? keys[p] : N;
  const uint2 val = valid ? vals[p] : make_uint2(0, 0);
  const uint32_t prev_edge = (lane == 0 && p > 0 && valid) ? keys[p - 1] : 0xFFFFFFFFu;
  const int64_t pl = chunk * WAVE + WAVE;  // first pair of the next chunk
  const uint32_t next_edge = (lane == WAVE - 1 && pl < n) ? keys[pl] : 0xFFFFFFFFu;
  const uint32_t up = __shfl_up(key, 1);
  const uint32_t down = __shfl_down(key, 1);
  const bool head = (lane == 0) ? (p == 0 || prev_edge != key) : (up != key);
  const bool tail = (lane == WAVE - 1) ? (next_edge != key) : (down != key);
  const bool live = valid && key < N;
  // head flags of the segmented scan (shared by every column group)
  bool seen = head;
  {
    bool f = head;
#pragma unroll
    for (int off = 1; off < WAVE; off <<= 1) {
      const bool fo = __shfl_up((int)f, off) != 0;
      if (lane >= off) f = f || fo;
    }
    seen = f;  // a head of this lane's run lies inside the chunk at or before this lane
  }
  const bool writer = live && (tail || lane == WAVE - 1);
  const bool partial = !seen || (lane == WAVE - 1 && !tail);
  const float wgt = __uint_as_float(val.y);
  const float* gp = gout + (size_t)val.x * M;
  float* dst = gtab + (size_t)key * M;
#pragma unroll 1
  for (int c0 = 0; c0 < M; c0 += 16) {
    float v[16];
#pragma unroll
    for (int e = 0; e < 16; e += 4) {
      const float4 g = live ? *reinterpret_cast<const float4*>(gp + c0 + e) : make_float4(0, 0, 0, 0);
      v[e] = wgt * g.x; v[e + 1] = wgt * g.y; v[e + 2] = wgt * g.z; v[e + 3] = wgt * g.w;
    }
    bool f = head;
#pragma unroll
    for (int off = 1; off < WAVE; off <<= 1) {
      const bool fo = __shfl_up((int)f, off) != 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float o = __shfl_up(v[e], off);
        if (lane >= off && !f) v[e] += o;
      }
      if (lane >= off) f = f || fo;
    }
    if (writer) {
      if (partial) {
#pragma unroll
        for (int e = 0; e < 16; ++e) unsafeAtomicAdd(dst + c0 + e, v[e]);
      } else {
#pragma unroll
        for (int e = 0; e < 16; e += 4) {
          float4* d4 = reinterpret_cast<float4*>(dst + c0 + e);
          float4 o = *d4;
          o.x += v[e]; o.y += v[e + 1]; o.z += v[e + 2]; o.w += v[e + 3];
          *d4 = o;
        }
      }
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
    if (K[i] < 2 || (K[i] & 1)) return LRAM_EBADK;
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
  }
  P->N = (uint32_t)N;
  P->L = *L;
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

unsigned grid_for(int64_t L) { return (unsigned)((L + THREADS - 1) / THREADS); }

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
  static int go(const float* q, const Params& P, const void* table, void* out, hipStream_t s) {
    hipLaunchKernelGGL((k_forward<DT, M>), dim3(grid_for(P.L)), dim3(THREADS), 0, s, q, P, table, out);
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

template <int DT, int M>
struct BwdAtomicLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                hipStream_t s) {
    hipLaunchKernelGGL((k_backward<DT, M, false>), dim3(grid_for(P.L)), dim3(THREADS), 0, s, q, P, table, g,
                       gt, gq, (uint32_t*)nullptr, (uint2*)nullptr);
    return launched();
  }
};

template <int DT, int M>
struct BwdSortedLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const SortWs& ws, hipStream_t s) {
    hipLaunchKernelGGL((k_backward<DT, M, true>), dim3(grid_for(P.L)), dim3(THREADS), 0, s, q, P, table, g, gt,
                       gq, ws.k0, ws.v0);
    int rc = launched();
    if (rc || !gt) return rc;
    int bits = 0;
    while (bits < 32 && (P.N >> bits) != 0) ++bits;  // keys lie in [0, N]
    uint32_t* kin = ws.k0;
    uint32_t* kout = ws.k1;
    uint2* vin = ws.v0;
    uint2* vout = ws.v1;
    for (int shift = 0; shift < bits; shift += RADIX_BITS) {
      hipLaunchKernelGGL(k_radix_hist, dim3(ws.nblocks), dim3(THREADS), 0, s, kin, ws.n, shift, ws.hist,
                         ws.nblocks);
      hipLaunchKernelGGL(k_scan_blocks, dim3((unsigned)ws.nbt), dim3(THREADS), 0, s, ws.hist, ws.nh, ws.totals);
      hipLaunchKernelGGL(k_scan_totals, dim3(1), dim3(THREADS), 0, s, ws.totals, ws.nbt);
      hipLaunchKernelGGL(k_scan_add, dim3((unsigned)ws.nbt), dim3(THREADS), 0, s, ws.hist, ws.nh, ws.totals);
      hipLaunchKernelGGL(k_radix_scatter, dim3(ws.nblocks), dim3(THREADS), 0, s, kin, vin, ws.n, shift, ws.hist,
                         ws.nblocks, kout, vout);
      if ((rc = launched())) return rc;
      std::swap(kin, kout);
      std::swap(vin, vout);
    }
    const unsigned chunks = (unsigned)((ws.n + WAVE - 1) / WAVE);
    hipLaunchKernelGGL((k_segreduce<M>), dim3((chunks + WAVES - 1) / WAVES), dim3(THREADS), 0, s, kin, vin, ws.n,
                       P.N, g, gt);
    return launched();
  }
};

}  // namespace

extern "C" {

int lram_version(void) { return 100; }

const char* lram_strerror(int status) {
  switch (status) {
    case LRAM_OK: return "ok";
    case LRAM_EINVAL: return "invalid argument (null/misaligned pointer or negative size)";
    case LRAM_EBADK: return "invalid torus: every K_i must be even and >= 2, N = prod K_i < 2^31";
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
  hipLaunchKernelGGL(k_neighbors, dim3(grid_for(L)), dim3(THREADS), 0, (hipStream_t)stream, q, P, slot, w, d2);
  return launched();
}

int lram_forward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                 int64_t N, int32_t m, void* out, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!out || (reinterpret_cast<uintptr_t>(out) & 15)) return LRAM_EINVAL;
  return dispatch<FwdLaunch>(dtype, m, q, P, table, out, (hipStream_t)stream);
}

int lram_backward_workspace_bytes(int64_t B, int64_t H, int32_t m, int mode, size_t* bytes) {
  if (!bytes || B < 0 || H < 0) return LRAM_EINVAL;
  if (m != 32 && m != 64) return LRAM_EDTYPE;
  if (mode == LRAM_SCATTER_ATOMIC) {
    *bytes = 0;
    return LRAM_OK;
  }
  if (mode == LRAM_SCATTER_SORTED) {
    if (H != 0 && B > INT64_MAX / H / NB) return LRAM_EINVAL;
    *bytes = sort_ws_layout(B * H, nullptr, nullptr);
    return LRAM_OK;
  }
  return LRAM_EMODE;
}

int lram_backward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, int mode,
                  void* workspace, size_t ws_bytes, void* stream) {
  (void)workspace;
  (void)ws_bytes;
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if (mode != LRAM_SCATTER_ATOMIC && mode != LRAM_SCATTER_SORTED) return LRAM_EMODE;
  if (L == 0) return LRAM_OK;
  if (!grad_out || (reinterpret_cast<uintptr_t>(grad_out) & 15)) return LRAM_EINVAL;
  if (!grad_table && !grad_q) return LRAM_EINVAL;
  if (grad_table && (reinterpret_cast<uintptr_t>(grad_table) & 15)) return LRAM_EINVAL;
  if (mode == LRAM_SCATTER_ATOMIC)
    return dispatch<BwdAtomicLaunch>(dtype, m, q, P, table, grad_out, grad_table, grad_q, (hipStream_t)stream);
  if (L > INT64_MAX / NB || L * NB >= (int64_t(1) << 32)) return LRAM_EINVAL;  // positions are 32-bit
  const size_t need = sort_ws_layout(L, nullptr, nullptr);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LRAM_EWORKSPACE;
  SortWs ws;
  sort_ws_layout(L, &ws, reinterpret_cast<char*>(workspace));
  return dispatch<BwdSortedLaunch>(dtype, m, q, P, table, grad_out, grad_table, grad_q, ws, (hipStream_t)stream);
}

}  // extern "C"
