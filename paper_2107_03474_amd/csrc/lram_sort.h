// lram_sort.h -- part of liblram (included by lram.hip only).
//
// Location sort: stable LSD radix sort and the segmented reduction of the
// sorted scatter.

#pragma once

namespace {

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
// addresses of a digit's output run.  V is the payload: the lookup index
// (uint32_t; IDENT: the first pass's payload is the element's own index, so it
// is never stored) or a (lookup, weight) pair (uint2).
template <typename V, bool IDENT>
__global__ void __launch_bounds__(THREADS) k_radix_scatter(const uint32_t* __restrict__ kin,
                                                           const V* __restrict__ vin, int64_t n, int shift,
                                                           const uint32_t* __restrict__ offs, int nblocks,
                                                           uint32_t* __restrict__ kout, V* __restrict__ vout) {
  static_assert(!IDENT || sizeof(V) == 4, "identity payloads are lookup indices");
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
      if constexpr (IDENT)
        vout[pos] = (V)(base + src);
      else
        vout[pos] = vin[base + src];
    }
  }
}

// Segmented reduction of the sorted pairs, bit-reproducible.  A group of M
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
                                                       const float* __restrict__ gout, float* __restrict__ gtab,
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
      g[u] = k[u] < N ? gout[(size_t)v.x * M + col] : 0.0f;
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
