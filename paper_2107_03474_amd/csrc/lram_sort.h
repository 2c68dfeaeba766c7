// lram_sort.h -- part of liblram (included by lram.hip only).
//
// Location sort: stable LSD radix sort and the segmented reduction of the
// sorted scatter.

#pragma once

namespace {

// Sorted value-gradient scatter: a stable LSD radix sort of the (location,
// (lookup, weight)) pairs by location, then a segmented reduction that writes
// every touched gradient row with one read-modify-write.  The same sort orders
// the lookups by closest point (lram_order).

constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;
constexpr int SORT_PASSES_MAX = 4;                 // keys are below 2^32
constexpr int SORT_ROUNDS = 16;                    // elements per thread per tile
constexpr int SORT_TILE = THREADS * SORT_ROUNDS;   // 4096
constexpr int SORT_WAVE_ELEMS = WAVE * SORT_ROUNDS;
static_assert(RADIX == THREADS, "one thread per digit");

// Count states of the single-pass scatter's look-back: a flag in the top two
// bits (0: not yet published), a digit count below.  32-bit states hold
// counts below 2^30 (sorts of fewer than 2^30 elements) and are read 24 to a
// look-back step; 64-bit states hold any 32-bit count, 16 to a step.
template <typename S>
struct CountState;
template <>
struct CountState<uint32_t> {
  static constexpr uint32_t AGGREGATE = 1u << 30;  // the tile's (group's) own count
  static constexpr uint32_t PREFIX = 2u << 30;     // count of this and every earlier tile (group)
  static constexpr uint32_t FLAGS = 3u << 30;
  static constexpr uint32_t VALUE = (1u << 30) - 1;
  static constexpr int BATCH = 24;
};
template <>
struct CountState<uint64_t> {
  static constexpr uint64_t AGGREGATE = 1ull << 62;
  static constexpr uint64_t PREFIX = 2ull << 62;
  static constexpr uint64_t FLAGS = 3ull << 62;
  static constexpr uint64_t VALUE = 0xFFFFFFFFull;
  static constexpr int BATCH = 16;
};
constexpr int64_t SORT_SMALL_STATES = int64_t(1) << 30;  // sorts below this many elements use 32-bit states
// Polls of a predecessor's state before a tile gives up (sets *fail; never
// expected: workgroups are dealt round-robin to the XCDs and each XCD starts
// its share in index order, so a tile waits only on lower tiles that are
// running or done, and those wait on nothing higher).
constexpr uint32_t LOOKBACK_POLLS = 1u << 22;

// Tiles per look-back group.
constexpr int LOOKBACK_GROUP = 32;
// Sort scratch cleared before every sort: global digit counts in
// SORT_HIST_COPIES copies [copy][pass][RADIX] (workgroup b adds into copy b %
// SORT_HIST_COPIES: atomics on one address serialise in memory, about 35 ns
// each), the failure word, the lookup order's gate-count partials
// [COUNT_COPIES], one to a 128-byte line (atomics on one line serialise
// too); then the tile states.
constexpr int SORT_HIST_COPIES = 16;
constexpr int SORT_FAIL = SORT_HIST_COPIES * SORT_PASSES_MAX * RADIX;
constexpr int SORT_COUNT = SORT_FAIL + 64;
constexpr int COUNT_COPIES = 64;
constexpr int COUNT_STRIDE = 32;  // words between gate-count partials
constexpr int SORT_HDR_WORDS = SORT_COUNT + COUNT_COPIES * COUNT_STRIDE;
static_assert((SORT_COUNT * 4) % 128 == 0, "gate-count partials start on a line");

__global__ void __launch_bounds__(THREADS) k_zero_words(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * THREADS) p[i] = 0u;
}

// Global digit counts of every pass: ghist[copy][p][d] summed over the copies
// is the number of keys whose digit p is d.  Each workgroup counts one
// contiguous chunk in LDS (per-wave counters, so fewer LDS atomics collide)
// and adds its nonzero bins to its copy.
__global__ void __launch_bounds__(THREADS) k_digit_hist(const uint32_t* __restrict__ keys, int64_t n, int passes,
                                                        uint32_t* __restrict__ ghist) {
  __shared__ uint32_t h[WAVES][SORT_PASSES_MAX][RADIX];
  const int t = threadIdx.x, w = t / WAVE;
#pragma unroll
  for (int k = 0; k < WAVES; ++k)
#pragma unroll
    for (int p = 0; p < SORT_PASSES_MAX; ++p) h[k][p][t] = 0;
  __syncthreads();
  const int64_t chunk = (n + gridDim.x - 1) / gridDim.x;
  const int64_t b = (int64_t)blockIdx.x * chunk, e = min<int64_t>(n, b + chunk);
  for (int64_t i = b + t; i < e; i += THREADS) {
    const uint32_t k = keys[i];
#pragma unroll
    for (int p = 0; p < SORT_PASSES_MAX; ++p)
      if (p < passes) atomicAdd(&h[w][p][(k >> (p * RADIX_BITS)) & (RADIX - 1)], 1u);
  }
  __syncthreads();
  uint32_t* g = ghist + (blockIdx.x % SORT_HIST_COPIES) * (SORT_PASSES_MAX * RADIX);
#pragma unroll
  for (int p = 0; p < SORT_PASSES_MAX; ++p) {
    const uint32_t c = h[0][p][t] + h[1][p][t] + h[2][p][t] + h[3][p][t];
    if (p < passes && c) atomicAdd(&g[p * RADIX + t], c);
  }
}

// Exclusive prefix sum of x over the workgroup's threads (thread t holds
// entry t); `part` is WAVES words of LDS.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* part) {
  const int w = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const uint32_t inc = wave_inclusive_scan(x);
  if (lane == WAVE - 1) part[w] = inc;
  __syncthreads();
  uint32_t pre = 0;
#pragma unroll
  for (int k = 0; k < WAVES; ++k) pre += k < w ? part[k] : 0u;
  return pre + inc - x;
}

// Sum of the count states state[i * RADIX + t], i = first .. last - 1 (digit
// t), read nearest first, BATCH at a time; a state not yet
// published is polled again.  STOP: the walk ends at the first PREFIX state
// (included), which holds the total of every state before it.
template <typename S, bool STOP, int BATCH>
__device__ __forceinline__ uint32_t lookback_sum(const S* __restrict__ state, int64_t first, int64_t last, int t,
                                                 uint32_t* __restrict__ fail) {
  using C = CountState<S>;
  uint32_t sum = 0;
  int64_t j = last - 1;  // nearest state not yet added
  uint32_t polls = 0;
  bool done = j < first;
  while (!done) {
    S v[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k)
      v[k] = j - k >= first ? __hip_atomic_load(state + (j - k) * RADIX + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                            : C::PREFIX;
    int used = 0;
    bool waiting = false;
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      if (!done && !waiting) {
        const S f = v[k] & C::FLAGS;
        if (f == 0) {
          waiting = true;
        } else {
          sum += (uint32_t)(v[k] & C::VALUE);
          ++used;
          done = (STOP && f == C::PREFIX) || j - k - 1 < first;
        }
      }
    }
    j -= used;
    if (waiting) {
      if (++polls > LOOKBACK_POLLS) {
        atomicOr(fail, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  return sum;
}

// One pass of a stable LSD radix sort in a single kernel: workgroup b takes
// tile b of SORT_TILE elements (no ticket: one atomic counter shared by every
// workgroup would start them about 35 ns apart), ranks them by digit inside
// each wave (8-ballot match, per-wave digit counters), publishes its digit
// counts, and finds how many elements of each digit the tiles before it hold
// with a two-level decoupled look-back: the tiles before it in its group of
// LOOKBACK_GROUP (their counts), then the groups before its own (the last tile
// of each group publishes the group's count, then the group's running total,
// walking back over groups until one whose total is known).  Every wait is on
// a lower tile.  It then writes its elements to their final positions through
// an LDS staging copy in digit order (keys, then payloads, through one
// buffer), so that consecutive threads store consecutive positions.  Element
// order inside a tile is index order (wave, round, lane), so equal digits keep
// their input order.  gcount: this pass's global digit counts
// (SORT_HIST_COPIES copies, SORT_PASSES_MAX * RADIX words apart); state:
// [tiles + groups][RADIX] cleared count states S (tiles, then groups).  V is
// the payload: the lookup index (IDENT: the element's own index, never read)
// or a (lookup, weight) pair (uint2).
template <typename V, bool IDENT, typename S>
__global__ void __launch_bounds__(THREADS, 4) k_onesweep(const uint32_t* __restrict__ kin, const V* __restrict__ vin,
                                                      int64_t n, int shift, const uint32_t* __restrict__ gcount,
                                                      S* __restrict__ state, uint32_t* __restrict__ fail,
                                                      uint32_t* __restrict__ kout, V* __restrict__ vout) {
  static_assert(!IDENT || sizeof(V) == 4, "identity payloads are lookup indices");
  using C = CountState<S>;
  // look-back step: 8-byte payloads keep twice the registers across it
  constexpr int LB = sizeof(V) > 4 ? 16 : C::BATCH;
  __shared__ uint32_t wcnt[WAVES][RADIX];  // per-wave digit counts, then the wave's start inside the digit
  __shared__ uint32_t dstart[RADIX];       // tile-local start of each digit
  __shared__ uint32_t gstart[RADIX];       // output position of the tile's first element of each digit
  __shared__ uint32_t part[2][WAVES];
  __shared__ V stage[SORT_TILE];           // keys, then payloads, in digit order
  const int t = threadIdx.x, w = t / WAVE, lane = t % WAVE;
#pragma unroll
  for (int k = 0; k < WAVES; ++k) wcnt[k][t] = 0;
  __syncthreads();
  const int64_t tile = blockIdx.x, tiles = gridDim.x;
  const int64_t base = tile * SORT_TILE;
  const int cnt = (int)min<int64_t>(SORT_TILE, n - base);
  uint32_t key[SORT_ROUNDS];
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = w * SORT_WAVE_ELEMS + r * WAVE + lane;
    key[r] = j < cnt ? kin[base + j] : 0u;
  }
  // rank inside the wave: earlier rounds' count of the digit + lanes below
  // with the same digit in this round
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (WAVE - lane));
  uint32_t slot[SORT_ROUNDS];  // digit | rank inside the wave << 8
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = w * SORT_WAVE_ELEMS + r * WAVE + lane;
    const bool valid = j < cnt;
    const uint32_t d = (key[r] >> shift) & (RADIX - 1);
    uint64_t match = __ballot(valid);
#pragma unroll
    for (int b = 0; b < RADIX_BITS; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bb = __ballot(bit);
      match &= bit ? bb : ~bb;
    }
    const uint32_t rank = (uint32_t)__popcll(match & lt);
    const uint32_t before = valid ? wcnt[w][d] : 0u;
    wave_lds_sync();
    if (valid && rank == 0) wcnt[w][d] = before + (uint32_t)__popcll(match);
    wave_lds_sync();
    slot[r] = d | ((before + rank) << 8);
  }
  __syncthreads();
  // thread t = digit t: the waves' starts inside the digit, the tile's count
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < WAVES; ++k) {
    const uint32_t x = wcnt[k][t];
    wcnt[k][t] = c;
    c += x;
  }
  S* tstate = state;                    // [tiles][RADIX]: AGGREGATE | count
  S* gstate = state + tiles * RADIX;    // [groups][RADIX]
  __hip_atomic_store(tstate + tile * RADIX + t, C::AGGREGATE | (S)c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // the payloads are loaded now, so that the ranking above had the memory
  // system to the keys alone and the loads overlap the look-back
  V val[IDENT ? 1 : SORT_ROUNDS];  // IDENT: the payload is formed when it is staged
  if constexpr (!IDENT) {
#pragma unroll
    for (int r = 0; r < SORT_ROUNDS; ++r) {
      const int j = w * SORT_WAVE_ELEMS + r * WAVE + lane;
      val[r] = j < cnt ? vin[base + j] : V{};
    }
  }
  dstart[t] = block_exclusive_scan(c, part[1]);
  __syncthreads();
  // each element's position in the tile's digit order (two 12-bit positions
  // to a register); stage the keys there (their registers are free during the
  // look-back)
  uint32_t pos2[SORT_ROUNDS / 2];
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const uint32_t d = slot[r] & (RADIX - 1);
    const uint32_t p = dstart[d] + wcnt[w][d] + (slot[r] >> 8);
    if (w * SORT_WAVE_ELEMS + r * WAVE + lane < cnt) reinterpret_cast<uint32_t*>(stage)[p] = key[r];
    if (r % 2 == 0)
      pos2[r / 2] = p & 0xFFFFu;
    else
      pos2[r / 2] |= p << 16;
  }
  const int64_t g = tile / LOOKBACK_GROUP, first = g * LOOKBACK_GROUP;
  const uint32_t intra = lookback_sum<S, false, LB>(tstate, first, tile, t, fail);
  const bool group_last = tile == min<int64_t>(first + LOOKBACK_GROUP, tiles) - 1;
  S* gs = gstate + g * RADIX + t;
  if (group_last)
    __hip_atomic_store(gs, (g == 0 ? C::PREFIX : C::AGGREGATE) | (S)(intra + c), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  const uint32_t before_group = lookback_sum<S, true, LB>(gstate, 0, g, t, fail);
  if (group_last && g > 0)
    __hip_atomic_store(gs, C::PREFIX | (S)(before_group + intra + c), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  uint32_t gc = 0;
#pragma unroll
  for (int k = 0; k < SORT_HIST_COPIES; ++k) gc += gcount[k * (SORT_PASSES_MAX * RADIX) + t];
  gstart[t] = block_exclusive_scan(gc, part[0]) + before_group + intra;
  __syncthreads();
  // write the keys out; keep each position's digit (four to a register)
  uint32_t dig[SORT_ROUNDS / 4];
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = r * THREADS + t;
    uint32_t d = 0;
    if (j < cnt) {
      const uint32_t k = reinterpret_cast<const uint32_t*>(stage)[j];
      d = (k >> shift) & (RADIX - 1);
      const uint32_t o = gstart[d] + (uint32_t)j - dstart[d];
      if (o < n)  // always, unless the look-back gave up
        kout[o] = k;
    }
    if (r % 4 == 0) dig[r / 4] = 0;
    dig[r / 4] |= d << (8 * (r % 4));
  }
  __syncthreads();
  // then the payloads through the same buffer
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = w * SORT_WAVE_ELEMS + r * WAVE + lane;
    if (j < cnt) {
      V v;
      if constexpr (IDENT)
        v = (V)(base + j);
      else
        v = val[r];
      stage[(pos2[r / 2] >> (16 * (r % 2))) & 0xFFFFu] = v;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < SORT_ROUNDS; ++r) {
    const int j = r * THREADS + t;
    if (j < cnt) {
      const uint32_t d = (dig[r / 4] >> (8 * (r % 4))) & (RADIX - 1);
      const uint32_t o = gstart[d] + (uint32_t)j - dstart[d];
      if (o < n) vout[o] = stage[j];
    }
  }
}

// Segmented reduction of the sorted pairs, bit-reproducible (nl: lookups, the
// bound of the pairs' lookup indices).  A group of M
// lanes (lane = column of the gradient row) owns a span of consecutive pairs
// (256, fewer for small batches so that every CU gets work) and walks it in
// order, prefetching 16 pairs and their upstream-gradient rows at a time; it
// accumulates w * G[lookup] while the location stays the same.  A run of one
// location that lies inside the span is written with one plain
// read-modify-write (no other group touches that row).  The partial sums of
// runs cut by the span's edges go to the span's two edge rows instead (head:
// the run that began in an earlier span, or the whole span when one run
// passes through it; tail: the run that begins here and continues), and
// k_segfix adds them in span order, one owner per cut run -- so every row's
// sum is formed in the same order on every call.
constexpr int SEG_SPAN = 256;
constexpr int SEG_BATCH = 16;
constexpr uint32_t SEG_HEAD = 1u;     // edge row 0 holds the partial of a run that began earlier
constexpr uint32_t SEG_TAIL = 2u;     // edge row 1 holds the partial of a run that began here and continues
constexpr uint32_t SEG_THROUGH = 4u;  // one run covers the whole span and continues past it (partial in row 0)

template <int M>
__global__ void __launch_bounds__(THREADS) k_segreduce(const uint32_t* __restrict__ keys,
                                                       const uint2* __restrict__ vals, int64_t n, uint32_t N,
                                                       uint32_t nl, const float* __restrict__ gout,
                                                       float* __restrict__ gtab,
                                                       int span, float* __restrict__ edge, uint32_t* __restrict__ flags) {
  const int64_t group = ((int64_t)blockIdx.x * THREADS + threadIdx.x) / M;
  const int col = threadIdx.x % M;
  const int64_t b = group * span;
  if (b >= n) return;
  const int64_t e = min<int64_t>(n, b + span);
  uint32_t cur = keys[b];
  uint32_t fl = 0;
  if (cur >= N) {  // padding sorts last
    if (col == 0) flags[group] = 0;
    return;
  }
  const bool head_cut = b > 0 && keys[b - 1] == cur;
  bool first = true;  // the current run is the span's first
  float acc = 0.0f;
  bool pad = false;   // reached the padding (key N), which sorts last
  float* erow = edge + (size_t)group * 2 * M + col;
  for (int64_t p = b; p < e && !pad; p += SEG_BATCH) {
    uint32_t k[SEG_BATCH];
    float wv[SEG_BATCH], g[SEG_BATCH];
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      const int64_t q = p + u;
      k[u] = q < e ? keys[q] : N;
      const uint2 v = q < e ? vals[q] : make_uint2(0, 0);
      wv[u] = __uint_as_float(v.y);
      g[u] = (k[u] < N && v.x < nl) ? gout[(size_t)v.x * M + col] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < SEG_BATCH; ++u) {
      if (p + u < e && !pad) {
        if (k[u] >= N) {
          pad = true;  // the current run ended just before the padding
        } else {
          if (k[u] != cur) {
            // the run of cur ended inside the span
            if (first && head_cut) {
              erow[0] = acc;
              fl |= SEG_HEAD;
            } else {
              gtab[(size_t)cur * M + col] += acc;
            }
            first = false;
            cur = k[u];
            acc = 0.0f;
          }
          acc = fmaf(wv[u], g[u], acc);
        }
      }
    }
  }
  // the span's last run: cut by the end unless the padding or the batch end
  // follows it
  const bool tail_cut = !pad && e < n && keys[e] == cur;
  if (first && head_cut) {
    erow[0] = acc;
    fl |= tail_cut ? (SEG_HEAD | SEG_THROUGH) : SEG_HEAD;
  } else if (tail_cut) {
    erow[M] = acc;
    fl |= SEG_TAIL;
  } else {
    gtab[(size_t)cur * M + col] += acc;
  }
  if (col == 0) flags[group] = fl;
}

// Runs cut by span edges: the span where a run begins (SEG_TAIL) adds, in span
// order, its tail partial, the partials of the spans the run passes through
// and the head partial of the span where it ends, and writes the row once
// (plain read-modify-write: no other group touches it).
template <int M>
__global__ void __launch_bounds__(THREADS) k_segfix(const uint32_t* __restrict__ keys, int64_t n, int span,
                                                    const float* __restrict__ edge, const uint32_t* __restrict__ flags,
                                                    int64_t groups, float* __restrict__ gtab) {
  const int64_t group = ((int64_t)blockIdx.x * THREADS + threadIdx.x) / M;
  const int col = threadIdx.x % M;
  if (group >= groups || !(flags[group] & SEG_TAIL)) return;
  const uint32_t key = keys[min<int64_t>(n, (group + 1) * span) - 1];
  float acc = edge[(size_t)group * 2 * M + M + col];
  for (int64_t g = group + 1; g < groups; ++g) {
    acc += edge[(size_t)g * 2 * M + col];
    if (!(flags[g] & SEG_THROUGH)) break;
  }
  gtab[(size_t)key * M + col] += acc;
}

}  // namespace
