// lram_merge.h -- part of liblram (included by lram.hip only).
//
// Batch-merged scatter: closest-point keys, the activation layer's
// coordinates, the merge gate and the fused search + per-batch merge kernel.

#pragma once

namespace {

// ---------------------------------------------------------------------------
// Batch-merged scatter.  Lookups whose queries share the closest lattice point
// share most of their neighbours; the lookups are ordered by that point's
// location (radix sort above), the backward emits (location, w) pairs in that
// order, and each batch of consecutive lookups (64; fewer for lists longer
// than 32, see merge_t) is reduced in LDS to one fp32 atomic row per distinct
// location of the batch.

// Location of the closest point of Lambda to the query qq (N for a
// non-finite query).
__device__ __forceinline__ uint32_t cell_location(const float (&qq)[8], const Params P) {
  float x[8];
  int c[8];
  if (!closest_point(qq, true, P, x, c)) return P.N;
  const int eps = c[0] & 1;
  uint32_t acc = eps ? P.N : 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    // |x_i| < 2 K_i and |x_i - c_i| <= 1 put y within [-K_i - 1, K_i]: two
    // periods up or one down bring it into [0, K_i) (K_i = 2 included)
    int y = (c[i] - eps) >> 1;
    y += y < 0 ? P.K[i] : 0;
    y += y < 0 ? P.K[i] : 0;
    y -= y >= P.K[i] ? P.K[i] : 0;
    acc += (uint32_t)y * P.S[i];
  }
  return acc >> 1;
}

// key[l] = cell_location of lookup l, and the digit counts of the keys for
// the first `passes` passes of the radix sort that orders them (as
// k_digit_hist: each workgroup counts one contiguous chunk of lookups in
// per-wave LDS counters and adds its nonzero bins to copy blockIdx %
// SORT_HIST_COPIES of ghist, cleared).  The workgroups also clear the sort's
// look-back states, clear[0, nclear), which no pass reads before this kernel
// ends.  Each lookup's input is loaded one lookup ahead.
template <bool TH>
__global__ void __launch_bounds__(THREADS) k_cell_key(const float* __restrict__ q, Params P,
                                                      uint32_t* __restrict__ key, int passes,
                                                      uint32_t* __restrict__ ghist, uint32_t* __restrict__ clear,
                                                      int64_t nclear) {
  __shared__ uint32_t h[WAVES][SORT_PASSES_MAX][RADIX];
  const int t = threadIdx.x, w = t / WAVE;
#pragma unroll
  for (int k = 0; k < WAVES; ++k)
#pragma unroll
    for (int p = 0; p < SORT_PASSES_MAX; ++p) h[k][p][t] = 0;
  for (int64_t i = (int64_t)blockIdx.x * THREADS + t; i < nclear; i += (int64_t)gridDim.x * THREADS) clear[i] = 0u;
  __syncthreads();
  const int64_t chunk = (P.L + gridDim.x - 1) / gridDim.x;
  const int64_t b = (int64_t)blockIdx.x * chunk, e = min<int64_t>(P.L, b + chunk);
  float4 v[in_vec4<TH>()];
  if (b + t < e) load_input<TH>(q + (b + t) * in_stride<TH>(), v);
  for (int64_t l = b + t; l < e; l += THREADS) {
    float4 cur[in_vec4<TH>()];
#pragma unroll
    for (int k = 0; k < in_vec4<TH>(); ++k) cur[k] = v[k];
    if (l + THREADS < e) load_input<TH>(q + (l + THREADS) * in_stride<TH>(), v);
    float qq[8], scale;
    query_from<TH>(cur, P, qq, scale);
    const uint32_t loc = cell_location(qq, P);
    key[l] = loc;
#pragma unroll
    for (int p = 0; p < SORT_PASSES_MAX; ++p)
      if (p < passes) atomicAdd(&h[w][p][(loc >> (p * RADIX_BITS)) & (RADIX - 1)], 1u);
  }
  __syncthreads();
  uint32_t* g = ghist + (blockIdx.x % SORT_HIST_COPIES) * (SORT_PASSES_MAX * RADIX);
#pragma unroll
  for (int p = 0; p < SORT_PASSES_MAX; ++p) {
    const uint32_t c = h[0][p][t] + h[1][p][t] + h[2][p][t] + h[3][p][t];
    if (p < passes && c) atomicAdd(&g[p * RADIX + t], c);
  }
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

// Number of positions whose sorted key equals a neighbour's, in COUNT_COPIES
// partial counters COUNT_STRIDE words apart (workgroup b adds into copy b %
// COUNT_COPIES, cleared, so that few atomics meet on one line);
// k_count_finalize adds them up.
constexpr int COUNT_UNROLL = 4;  // positions per thread whose loads are issued together
__global__ void __launch_bounds__(THREADS) k_count_shared(const uint32_t* __restrict__ keys, int64_t L,
                                                          uint32_t* __restrict__ copies) {
  __shared__ uint32_t wsum[WAVES];
  constexpr int U = COUNT_UNROLL;
  uint32_t c = 0;
  const int64_t stride = (int64_t)gridDim.x * THREADS;
  for (int64_t i0 = (int64_t)blockIdx.x * THREADS + threadIdx.x; i0 < L; i0 += U * stride) {
    uint32_t kp[U], kc[U], kn[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      kc[u] = i < L ? keys[i] : 0u;
      kp[u] = i < L && i > 0 ? keys[i - 1] : ~kc[u];
      kn[u] = i + 1 < L ? keys[i + 1] : ~kc[u];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) c += (i0 + u * stride < L && (kp[u] == kc[u] || kn[u] == kc[u])) ? 1u : 0u;
  }
#pragma unroll
  for (int mask = 1; mask < WAVE; mask <<= 1) c += __shfl_xor(c, mask);
  if (threadIdx.x % WAVE == 0) wsum[threadIdx.x / WAVE] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t t = wsum[0] + wsum[1] + wsum[2] + wsum[3];
    if (t) atomicAdd(copies + (blockIdx.x % COUNT_COPIES) * COUNT_STRIDE, t);
  }
}

// count[0] = the sum of the partial counters, count[1] = the sort's failure
// word (one wave).
__global__ void k_count_finalize(const uint32_t* __restrict__ copies, const uint32_t* __restrict__ sort_fail,
                                 uint32_t* __restrict__ count) {
  uint32_t s = 0;
  for (int i = threadIdx.x; i < COUNT_COPIES; i += WAVE) s += copies[i * COUNT_STRIDE];
#pragma unroll
  for (int mask = 1; mask < WAVE; mask <<= 1) s += __shfl_xor(s, mask);
  if (threadIdx.x == 0) {
    count[0] = s;
    count[1] = *sort_fail;
  }
}

constexpr int64_t AUTO_MERGE_MIN = 131072;      // LRAM_SCATTER_AUTO merges from this many lookups on
constexpr int MERGE_P = 64 * NB;                // pair slots per batch
constexpr int MERGE_H = 2 * MERGE_P;            // hash entries (load factor <= 1/2)
constexpr int MERGE_HBITS = 12;
static_assert((1 << MERGE_HBITS) == MERGE_H, "hash size");
constexpr int MERGE_PPT = MERGE_P / THREADS;    // pair slots per thread
constexpr int MERGE_HPT = MERGE_H / THREADS;    // hash entries per thread (consecutive)
constexpr int32_t MERGE_EMPTY = -1;

// Pair layout of a batch.  Fixed: lookup b's list of KS entries (padding
// included) fills slots [b KS, (b+1) KS).  Compact (the untruncated lookup,
// whose lists are up to 241 long but 65 on average): each wave owns MERGE_SEG
// slots and appends its lookups' real pairs there; a lookup that no longer
// fits scatters with per-lookup atomics instead.
template <int KS>
constexpr bool merge_compact() { return KS == KALL; }
constexpr int MERGE_SEG = MERGE_P / WAVES;

// Lookups per batch (one workgroup) for lists of KS neighbours: 64, fewer for
// longer fixed lists so that a batch never holds more than MERGE_P pairs, 32
// for the compact layout.
template <int KS>
constexpr int merge_t() { return merge_compact<KS>() ? 32 : (KS <= NB ? 64 : MERGE_P / KS); }
template <int KS>
constexpr int merge_lpw() { return merge_t<KS>() / WAVES; }
static_assert(merge_t<16>() * 16 <= MERGE_P && merge_t<64>() * 64 <= MERGE_P && KALL <= MERGE_SEG, "batch sizes");
static_assert(MERGE_P < 65536, "batch-local positions are 16 bits wide");

// LDS of the fused kernel, two regions whose contents change from phase to phase.
// Region a: the batch's (location, w) pairs while the search runs; then the
// hash table's location tags; then, compacted to its front, the distinct
// locations in group order, with the pair weights in group order in its upper
// half.  Region b: the search; then the hash entries' pair counts (later their
// first positions in group order), the upstream gradient rows of the batch,
// the groups' first positions and the pairs' lookups in group order.
template <int M, int T>
struct alignas(16) MergeWork {
  uint32_t cnt[MERGE_H / 2];    // 16-bit pair count of each entry, then its first position in group order
  float g[T][M];                // upstream gradient rows of the batch
  uint16_t start[MERGE_P + 2];  // first position of each group (location) in group order
  uint8_t pt[MERGE_P];          // lookup (in the batch) of each pair, in group order
  uint32_t wsum[WAVES][2];
  uint32_t ngroups;
};

template <int M, int KS>
struct alignas(16) FusedLds {
  union {
    struct {
      int32_t loc[MERGE_P];     // (location, w) of every pair (-1: empty slot)
      float w[MERGE_P];
      uint8_t lk[merge_compact<KS>() ? MERGE_P : 1];  // compact layout: the pair's lookup in the batch
    } pairs;
    int32_t tag[MERGE_H];       // hash tags; then group locations [0, ngroups) and pair weights [MERGE_P, 2 MERGE_P)
  } a;
  union {
    SearchLds<merge_lpw<KS>(), KS> search;
    MergeWork<M, merge_t<KS>()> merge;
  } b;
};
static_assert(MERGE_H == 2 * MERGE_P, "group locations and pair weights share the tag array");

// Waves per SIMD that the LDS of one batch allows (160 KB per CU, 4 SIMDs):
// the register budget is held to it, so registers do not lower the occupancy
// below what the LDS permits -- except for fp32 tables with m = 64, whose
// 256-byte rows need more registers than four waves per SIMD leave.
template <int DT, int M, int KS>
constexpr int merge_waves_per_simd() {
  const int w = (int)((160 * 1024) / sizeof(FusedLds<M, KS>)) * WAVES / 4;
  return (DT == LRAM_F32 && M == 64 && w > 3) ? 3 : w;
}

// One workgroup = one batch of merge_t<KS>() consecutive positions of the
// order perm: each wave searches merge_lpw<KS>() lookups (with dq as in
// k_backward) and leaves their (location, w) pairs -- KS per lookup, padding
// included -- in LDS; then the workgroup hashes the pairs by location, lays
// them out grouped by location, and M lanes per distinct location sum w * G
// over its pairs and add the row with fp32 atomics.
// Several workgroups per CU overlap one's search with another's atomics.
// A batch in which fewer than a tenth of the lookups share their closest
// point with a neighbour in the order (queries spread thinly over the torus)
// has little to merge: it scatters with per-lookup atomics instead.
// SAVED: the forward's lists (NbrList saved) replace the search.
template <int DT, int M, bool TH, int KS = NB, bool SAVED = false>
__global__ void __launch_bounds__(THREADS, (merge_waves_per_simd<DT, M, KS>())) k_backward_merged(const float* __restrict__ q, Params P,
                                                             const void* __restrict__ table,
                                                             const float* __restrict__ gout,
                                                             float* __restrict__ gtab, float* __restrict__ gq,
                                                             const uint32_t* __restrict__ skey,
                                                             const uint32_t* __restrict__ perm,
                                                             const uint32_t* __restrict__ gate, NbrList saved) {
  __shared__ FusedLds<M, KS> S;
  if (!merge_chosen(*gate, P.L)) return;  // the batch is scattered by k_backward instead
  const int t = threadIdx.x, wave = t / WAVE, lane = t % WAVE;
  const int64_t bbase = xcd_block() * (WAVES * P.lpw);  // consecutive batches share an L2
  const int nt = (int)min<int64_t>(WAVES * P.lpw, P.L - bbase);
  bool shared = false;
  if (t < nt) {
    const uint32_t k = skey[bbase + t];
    shared = (t > 0 && skey[bbase + t - 1] == k) || (t + 1 < nt && skey[bbase + t + 1] == k);
  }
  const bool merge = 10 * __syncthreads_count(shared) >= nt;
  constexpr bool COMPACT = merge_compact<KS>();
  int used = 0;  // compact layout: slots of this wave's segment taken (wave-uniform)
  {
    const int64_t base = bbase + (int64_t)wave * P.lpw;
    const int nl = (int)max<int64_t>(0, min<int64_t>(P.lpw, P.L - base));
    if (nl > 0) {
      Search<KS> srch(P, S.b.search.tab, S.b.search.wave[wave], wave, lane);
      WaveLds<KS>& W = S.b.search.wave[wave];
      Frame* FR = S.b.search.frames[wave];
      const uint32_t my_l = phase_a_perm<TH>(q, perm, base, nl, P, FR, lane);
      const char* tb = reinterpret_cast<const char*>(table);
      for (int i = 0; i < nl; ++i) {
        const Frame& F = FR[i];
        const Sel sel = read_sel(F);
        const int64_t l = (int64_t)(uint32_t)__builtin_amdgcn_readlane(my_l, i);
        int count;
        if constexpr (SAVED)
          count = srch.load(F, sel, 0, saved, l, P.N);
        else
          count = srch.run(F, sel, 0);
        if (!merge && count > 0) scatter_atomic<M, KS>(W, count, gout, l, gtab, lane);
        if (gq && l < P.L) grad_query<DT, M, TH, KS>(F, W, S.b.search.tab, count, tb, gout, l, lane, gq, q, P);
        if (merge && !COMPACT) {
#pragma unroll
          for (int j = lane; j < KS; j += WAVE) {
            const int pidx = (wave * P.lpw + i) * KS + j;
            S.a.pairs.loc[pidx] = W.nbr[0][j].slot;
            S.a.pairs.w[pidx] = W.wgt[0][j];
          }
        }
        if constexpr (COMPACT) {
          if (merge && used + count <= MERGE_SEG) {
            for (int j = lane; j < count; j += WAVE) {
              const int pidx = wave * MERGE_SEG + used + j;
              S.a.pairs.loc[pidx] = W.nbr[0][j].slot;
              S.a.pairs.w[pidx] = W.wgt[0][j];
              S.a.pairs.lk[pidx] = (uint8_t)(wave * P.lpw + i);
            }
            used += count;
          } else if (merge && count > 0) {
            scatter_atomic<M, KS>(W, count, gout, l, gtab, lane);  // the segment is full
          }
        }
        wave_lds_sync();
      }
    }
  }
  if (!merge) return;  // uniform across the workgroup
  if constexpr (COMPACT) {
    for (int j = used + lane; j < MERGE_SEG; j += WAVE) S.a.pairs.loc[wave * MERGE_SEG + j] = -1;
  }
  __syncthreads();
  // this thread's pairs into registers: region a then takes the hash tags
  int32_t locv[MERGE_PPT];
  float wv[MERGE_PPT];
  uint8_t lkv[MERGE_PPT];
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) {
    const int pidx = k * THREADS + t;
    locv[k] = -1;
    wv[k] = 0.0f;
    lkv[k] = (uint8_t)(pidx / KS);
    if (pidx < (COMPACT ? MERGE_P : nt * KS)) {
      locv[k] = S.a.pairs.loc[pidx];
      wv[k] = S.a.pairs.w[pidx];
      if constexpr (COMPACT) lkv[k] = S.a.pairs.lk[pidx];
    }
  }
  __syncthreads();
  MergeWork<M, merge_t<KS>()>& MW = S.b.merge;
  int32_t* tag = S.a.tag;
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) tag[k * THREADS + t] = MERGE_EMPTY;
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) MW.cnt[k * THREADS + t] = 0u;
  for (int i = t; i < nt * (M / 4); i += THREADS) {
    const int r = i / (M / 4), c4 = i % (M / 4);
    const uint32_t l = perm[bbase + r];
    reinterpret_cast<float4*>(MW.g[r])[c4] =
        l < P.L ? reinterpret_cast<const float4*>(gout + (size_t)l * M)[c4] : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();
  // insert every pair's location; keep (entry, rank among the entry's pairs)
  uint32_t ent[MERGE_PPT];
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) {
    ent[k] = 0xFFFFFFFFu;
    const int32_t loc = locv[k];
    if (loc >= 0) {
      uint32_t h = ((uint32_t)loc * 0x9E3779B1u) >> (32 - MERGE_HBITS);
      while (true) {
        const int32_t old = atomicCAS(&tag[h], MERGE_EMPTY, loc);
        if (old == MERGE_EMPTY || old == loc) break;
        h = (h + 1) & (MERGE_H - 1);
      }
      const uint32_t sh = 16u * (h & 1u);
      const uint32_t rank = (atomicAdd(&MW.cnt[h >> 1], 1u << sh) >> sh) & 0xFFFFu;
      ent[k] = h | (rank << 16);
    }
  }
  __syncthreads();
  // exclusive scan over the entries: group index and first position of each
  // occupied entry (this thread owns entries [t*HPT, (t+1)*HPT)); the owned
  // tags are read now, before the group locations overwrite the front of the
  // tag array
  uint32_t c[MERGE_HPT];
  int32_t tg[MERGE_HPT];
  uint32_t ng = 0, np = 0;
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) {
    const uint32_t wd = MW.cnt[t * (MERGE_HPT / 2) + k];
    c[2 * k] = wd & 0xFFFFu;
    c[2 * k + 1] = wd >> 16;
  }
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) {
    tg[k] = tag[t * MERGE_HPT + k];
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
    MW.start[gb + ng] = (uint16_t)(pb + np);
  }
  uint32_t first[MERGE_HPT];
#pragma unroll
  for (int k = 0; k < MERGE_HPT; ++k) {
    first[k] = pb;
    if (c[k]) {
      tag[gb] = tg[k];  // group gb's location; gb <= entry index, every tag already read
      MW.start[gb] = (uint16_t)pb;
      ++gb;
      pb += c[k];
    }
  }
#pragma unroll
  for (int k = 0; k < MERGE_HPT / 2; ++k) MW.cnt[t * (MERGE_HPT / 2) + k] = first[2 * k] | (first[2 * k + 1] << 16);
  __syncthreads();
  // rows of 32 columns (one 128-byte line): fetch the line of every distinct
  // location's gradient row into L2 now, so that the atomics below find it
  // there (the values are not used: loads that nothing waits for until the
  // kernel's end).  Rows of 64 columns measured no gain from it.
  constexpr bool PREFETCH = M == 32;
  uint32_t pfv[MERGE_PPT];
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) pfv[k] = 0u;
  if constexpr (PREFETCH) {
    const uint32_t ng = MW.ngroups;
#pragma unroll
    for (int k = 0; k < MERGE_PPT; ++k) {
      const uint32_t gi = t + k * THREADS;
      if (gi < ng) pfv[k] = reinterpret_cast<const uint32_t*>(gtab)[(size_t)tag[gi] * M];
    }
  }
  // pairs into group order: weights in the upper half of the tag array
  float* pw = reinterpret_cast<float*>(tag + MERGE_P);
  uint8_t* pt = MW.pt;
#pragma unroll
  for (int k = 0; k < MERGE_PPT; ++k) {
    if (ent[k] != 0xFFFFFFFFu) {
      const uint32_t h = ent[k] & 0xFFFFu;
      const uint32_t pos = ((MW.cnt[h >> 1] >> (16u * (h & 1u))) & 0xFFFFu) + (ent[k] >> 16);
      pw[pos] = wv[k];
      pt[pos] = lkv[k];
    }
  }
  __syncthreads();
  // one row per distinct location: M lanes (lane = column) sum w * G over its
  // pairs.  A lane takes U locations at a time and reads their first pairs
  // together (most locations have one or two pairs), so those LDS reads
  // overlap; further pairs follow location by location.
  constexpr int GROUPS = THREADS / M;
  constexpr int U = 4;
  const int col = t % M;
  const uint32_t ngroups = MW.ngroups;
  for (uint32_t g0 = t / M; g0 < ngroups; g0 += U * GROUPS) {
    uint32_t p0[U], p1[U];
    int32_t loc[U];
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t gi = g0 + u * GROUPS;
      const bool ok = gi < ngroups;
      p0[u] = ok ? MW.start[gi] : 0u;
      p1[u] = ok ? MW.start[gi + 1] : 0u;
      loc[u] = ok ? tag[gi] : -1;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const uint32_t p = p0[u] < p1[u] ? p0[u] : 0u;
      acc[u] = fmaf(pw[p], MW.g[pt[p]][col], 0.0f);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      for (uint32_t p = p0[u] + 1; p < p1[u]; ++p) acc[u] = fmaf(pw[p], MW.g[pt[p]][col], acc[u]);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (loc[u] >= 0) unsafeAtomicAdd(gtab + (size_t)loc[u] * M + col, acc[u]);
  }
  if constexpr (PREFETCH) sink_prefetch(pfv, ngroups > (uint32_t)MERGE_P, gtab);
}

}  // namespace
