// lram_common.h -- part of liblram (included by lram.hip only).
//
// Constants, kernel parameters, LDS layouts and small device helpers shared by
// every kernel.

#pragma once

namespace {

constexpr int NB = LRAM_NEIGHBOURS;  // 32, Sec. 2.6
constexpr int WAVE = 64;
constexpr int WAVES = 4;                 // waves per workgroup
constexpr int THREADS = WAVE * WAVES;
constexpr int NS_STRICT = (E8_NSTRICT + WAVE - 1) / WAVE;      // 4 candidate slots per lane
constexpr int NS_BOUND = (E8_NBOUNDARY + WAVE - 1) / WAVE;     // 3
constexpr int NS_ALL = NS_STRICT + NS_BOUND;
constexpr int NS_FAST = E8_FAST / WAVE;                          // 3: the fast set's slots per lane
constexpr int NS_FAST2 = E8_FAST2 / WAVE;                        // 2: its first tier
static_assert(E8_FAST % WAVE == 0 && NS_FAST < NS_STRICT, "the fast candidate set fills whole slots");
static_assert(E8_FAST2 % WAVE == 0 && NS_FAST2 < NS_FAST, "the first tier fills whole slots");
constexpr int CMIN = E8_CAND_MIN;
constexpr int NV = E8_CAND_MAX - E8_CAND_MIN + 1;
static_assert(NV == 8, "each per-query table row holds the 8 possible candidate coordinate values");
static_assert(WAVES <= 4, "the wave index is folded into byte-sized LDS offsets");
constexpr int KMAX = 8192;  // per-coordinate torus side bound: lattice coordinates fit in int16
constexpr int XCDS = 8;  // accelerator complex dies of an MI355X
constexpr int64_t LMAX = (int64_t(1) << 31) - 1;  // lookups per call

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
// A query whose k-th closest candidate among the first E8_FAST lies below
// KEY_FAST takes its closest k from them: every later candidate lies at
// distance^2 >= E8_FAST_BOUND from F, and the reduction puts a query within
// about 1e-5 (in distance^2) of F, far inside the 2^-7 margin.  The same
// holds for the first E8_FAST2 candidates and KEY_FAST2, tried first.
constexpr uint32_t KEY_FAST = __builtin_bit_cast(uint32_t, E8_FAST_BOUND - 0.0078125f);
constexpr uint32_t KEY_FAST2 = __builtin_bit_cast(uint32_t, E8_FAST2_BOUND - 0.0078125f);

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

// Per-wave search state for lists of KS neighbours, NBUF lists deep (the k =
// 32 forward double-buffers them: lookup t+1 is searched while t is consumed).
template <int KS, int NBUF = 1>
struct alignas(16) WaveLds {
  Nbr nbr[NBUF][KS];
  float wgt[NBUF][KS];
  uint32_t tie[tie_max<KS>()][2];
  uint32_t hist[64];  // distance histogram of the selection, 64 buckets on [4, 8)
};

// Neighbour lists saved by the forward for the backward (any pointer null: no
// list).  Entry j of lookup l sits at [l][j] in the search's own order, padding
// included: slot (-1 for padding), weight, and code -- the point's coordinates
// p in the fundamental-region frame of its query (Sec. 2.6: k = c + sigma pi^-1 p),
// eight 3-bit fields p_r - CMIN, F position r in bits [3r, 3r + 3).
struct NbrList {
  int32_t* slot;
  float* w;
  uint32_t* code;
  __host__ __device__ bool on() const { return slot != nullptr; }
};

// Packed candidate bytes (4 (p_r - CMIN) + 64 w per F position) <-> code.
__device__ __forceinline__ uint32_t code_of(uint32_t lo, uint32_t hi) {
  auto squeeze = [](uint32_t v) {
    v = (v >> 2) & 0x07070707u;
    return (v & 0x7u) | ((v >> 5) & 0x38u) | ((v >> 10) & 0x1C0u) | ((v >> 15) & 0xE00u);
  };
  return squeeze(lo) | (squeeze(hi) << 12);
}
__device__ __forceinline__ void bytes_of(uint32_t code, uint32_t wbyte, uint32_t& lo, uint32_t& hi) {
  auto spread = [](uint32_t c) {
    return (c & 0x7u) | ((c & 0x38u) << 5) | ((c & 0x1C0u) << 10) | ((c & 0xE00u) << 15);
  };
  const uint32_t wb = wbyte * 0x01010101u;
  lo = (spread(code & 0xFFFu) << 2) + wb;
  hi = (spread((code >> 12) & 0xFFFu) << 2) + wb;
}

// per-query tables, [coordinate i][wave w][value v] -> byte i*256 + w*64 + 4v
struct alignas(16) Tables {
  float qt[8 * 64];
  uint32_t st[8 * 64];
  float et[8 * 64];
};

// LDS of the search for FR lookups per wave and lists of KS neighbours.
template <int FR, int KS = NB, int NBUF = 1>
struct alignas(16) SearchLds {
  Tables tab;
  WaveLds<KS, NBUF> wave[WAVES];
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

// Keeps prefetch loads (lines fetched into L2 ahead of atomics on them) alive:
// their values meet here only, in a store that never happens (never is a
// condition false whenever the kernel runs correctly).
template <int NP>
__device__ __forceinline__ void sink_prefetch(const uint32_t (&v)[NP], bool never, float* __restrict__ dst) {
  uint32_t x = 0;
#pragma unroll
  for (int k = 0; k < NP; ++k) x ^= v[k];
  if (never && x == 0x7FC00001u) dst[0] = 0.0f;
}

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

// Workgroup index remapped so that each XCD (the dispatcher deals consecutive
// workgroups round-robin over the 8 XCDs, each with its own L2) walks one
// contiguous range of the grid: a bijection on [0, gridDim.x).
__device__ __forceinline__ int64_t xcd_block() {
  const int64_t G = gridDim.x, b = blockIdx.x;
  const int64_t x = b % XCDS, j = b / XCDS, q = G / XCDS, r = G % XCDS;
  return x < r ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
}

}  // namespace
