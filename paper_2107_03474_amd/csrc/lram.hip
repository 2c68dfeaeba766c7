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

#include <mutex>
#include <utility>

#include "../../include/lram.h"
#include "e8_candidates.inc"

#include "lram_common.h"
#include "lram_search.h"
#include "lram_lookup.h"
#include "lram_backward.h"
#include "lram_sort.h"
#include "lram_merge.h"
#include "lram_train.h"

namespace {

// ---------------------------------------------------------------------------
// Host side.

thread_local int g_last_hip_error = 0;

// Alignment of the device pointers: 16 bytes where the kernels move 16-byte
// vectors, the element size for the per-element arrays.
bool misaligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }
bool misaligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3) != 0; }

int check_common(const float* q, int64_t B, int64_t H, const int32_t* K, int64_t* L, Params* P) {
  if (B < 0 || H < 0 || !K) return LRAM_EINVAL;
  if (H != 0 && B > INT64_MAX / H) return LRAM_EINVAL;
  *L = B * H;
  if (*L > LMAX) return LRAM_EINVAL;  // keeps every grid below 2^32 work-items
  int64_t N = 1;
  for (int i = 0; i < 8; ++i) {
    if (K[i] < 2 || (K[i] & 1) || K[i] > KMAX) return LRAM_EBADK;
    N *= K[i];
    if (N >= (int64_t(1) << 31)) return LRAM_EBADK;
  }
  if (*L > 0) {
    if (!q || misaligned16(q)) return LRAM_EINVAL;
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
  if (L > 0 && (!table || misaligned16(table))) return LRAM_EINVAL;
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
  static int go(const float* q, const Params& P, const void* table, void* out, bool th, const uint32_t* perm,
                NbrList save, hipStream_t s) {
    const dim3 g(grid_for(P)), b(THREADS);
    if (th)
      hipLaunchKernelGGL((k_forward<DT, M, true>), g, b, 0, s, q, P, table, out, perm, save);
    else if (perm && save.on())
      hipLaunchKernelGGL((k_forward<DT, M, false, true, true>), g, b, 0, s, q, P, table, out, perm, save);
    else if (perm)
      hipLaunchKernelGGL((k_forward<DT, M, false, true, false>), g, b, 0, s, q, P, table, out, perm, save);
    else if (save.on())
      hipLaunchKernelGGL((k_forward<DT, M, false, false, true>), g, b, 0, s, q, P, table, out, perm, save);
    else
      hipLaunchKernelGGL((k_forward<DT, M, false>), g, b, 0, s, q, P, table, out, perm, save);
    return launched();
  }
};

size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// Carves consecutive 256-byte aligned pieces out of a workspace (base = null:
// only counts the bytes).
struct Carver {
  char* base;
  size_t off = 0;
  char* take(size_t bytes) {
    char* ptr = base ? base + off : nullptr;
    off += align256(bytes);
    return ptr;
  }
};

// Radix-sort buffers for n keys with payloads of type V, ping-ponged between
// (ka, va) and (kb, vb), and the sort's scratch: hdr [SORT_HDR_WORDS] (global
// digit counts, failure word, gate-count partials) followed by the count
// states [SORT_PASSES_MAX][tiles + groups][RADIX], all cleared by the sort
// itself.
template <typename V>
struct Radix {
  uint32_t *ka, *kb;
  V *va, *vb;
  uint32_t* hdr;
  uint64_t* state;
  int64_t n;
  int64_t tiles;
  int64_t states;  // tiles + look-back groups
};

template <typename V>
void carve_radix_scratch(int64_t n, Carver& c, Radix<V>* r) {
  const int64_t tiles = (n + SORT_TILE - 1) / SORT_TILE;
  const int64_t states = tiles + (tiles + LOOKBACK_GROUP - 1) / LOOKBACK_GROUP;
  // hdr and the states are contiguous (SORT_HDR_WORDS * 4 is a multiple of 256)
  static_assert((SORT_HDR_WORDS * 4) % 256 == 0, "sort scratch layout");
  char* h = c.take((size_t)SORT_HDR_WORDS * 4);
  char* st = c.take((size_t)SORT_PASSES_MAX * states * RADIX * 8);
  if (r) {
    r->hdr = (uint32_t*)h;
    r->state = (uint64_t*)st;
    r->n = n;
    r->tiles = tiles;
    r->states = states;
  }
}

int radix_passes(uint32_t N) {
  int bits = 0;
  while (bits < 32 && (N >> bits) != 0) ++bits;
  return (bits + RADIX_BITS - 1) / RADIX_BITS;
}

// Stable LSD radix sort of the n (key, payload) pairs in (ka, va), keys in
// [0, N]: the result is in (ka, va) after an even number of passes and in
// (kb, vb) after an odd one.  IDENT: the payload of element i is i (va is
// not read).  Kernels: clear the scratch, count every pass's digits, then one
// single-pass scatter per digit.
template <typename V, bool IDENT, typename S>
int radix_passes_run(const Radix<V>& r, int passes, hipStream_t s) {
  uint32_t* kin = r.ka;
  uint32_t* kout = r.kb;
  V* vin = r.va;
  V* vout = r.vb;
  for (int p = 0; p < passes; ++p) {
    S* st = reinterpret_cast<S*>(r.state) + (int64_t)p * r.states * RADIX;
    const uint32_t* gc = r.hdr + p * RADIX;
    if (IDENT && p == 0)
      hipLaunchKernelGGL((k_onesweep<V, IDENT, S>), dim3((unsigned)r.tiles), dim3(THREADS), 0, s,
                         (const uint32_t*)kin, (const V*)vin, r.n, p * RADIX_BITS, gc, st, r.hdr + SORT_FAIL, kout,
                         vout);
    else
      hipLaunchKernelGGL((k_onesweep<V, false, S>), dim3((unsigned)r.tiles), dim3(THREADS), 0, s,
                         (const uint32_t*)kin, (const V*)vin, r.n, p * RADIX_BITS, gc, st, r.hdr + SORT_FAIL, kout,
                         vout);
    if (int rc = launched()) return rc;
    std::swap(kin, kout);
    std::swap(vin, vout);
  }
  return LRAM_OK;
}

// Stable LSD radix sort of the n (key, payload) pairs in (ka, va), keys in
// [0, N]: the result is in (ka, va) after an even number of passes and in
// (kb, vb) after an odd one.  IDENT: the payload of element i is i (va is
// not read).  Kernels: clear the scratch, count every pass's digits, then one
// single-pass scatter per digit (32-bit look-back states below 2^30 elements).
template <typename V, bool IDENT>
int radix_sort(const Radix<V>& r, uint32_t N, hipStream_t s) {
  if (r.n <= 0) return LRAM_OK;
  const int passes = radix_passes(N);
  const bool small = r.n < SORT_SMALL_STATES;
  const int64_t words = SORT_HDR_WORDS + (int64_t)passes * r.states * RADIX * (small ? 1 : 2);
  const int64_t zb = (words + THREADS - 1) / THREADS;
  hipLaunchKernelGGL(k_zero_words, dim3((unsigned)(zb < 1024 ? zb : 1024)), dim3(THREADS), 0, s, r.hdr, words);
  hipLaunchKernelGGL(k_digit_hist, dim3((unsigned)(r.tiles < 1024 ? r.tiles : 1024)), dim3(THREADS), 0, s,
                     (const uint32_t*)r.ka, r.n, passes, r.hdr);
  if (int rc = launched()) return rc;
  return small ? radix_passes_run<V, IDENT, uint32_t>(r, passes, s) : radix_passes_run<V, IDENT, uint64_t>(r, passes, s);
}

// The lookup order of lram_order, which is also the merged scatter's
// workspace: a 256-byte header (word 0: the merge gate's count of lookups that
// share their closest lattice point with a neighbour in the order), then the
// sorted keys [L] and positions [L] (sort.ka, sort.va: the documented
// offsets), then the sort's scratch.
struct OrderWs {
  uint32_t* shared;
  Radix<uint32_t> sort;
};

constexpr size_t ORDER_KEYS_OFFSET = 256;

size_t order_layout(int64_t L, OrderWs* o, char* base) {
  Carver c{base};
  char* hdr = c.take(ORDER_KEYS_OFFSET);
  char* ka = c.take(L * 4);
  char* va = c.take(L * 4);
  char* kb = c.take(L * 4);
  char* vb = c.take(L * 4);
  carve_radix_scratch<uint32_t>(L, c, o ? &o->sort : nullptr);
  if (o) {
    o->shared = (uint32_t*)hdr;
    o->sort.ka = (uint32_t*)ka;
    o->sort.va = (uint32_t*)va;
    o->sort.kb = (uint32_t*)kb;
    o->sort.vb = (uint32_t*)vb;
  }
  return c.off;
}

// Workspace of the sorted scatter: the sort of the 32 L (location, (lookup, w))
// pairs, and the segmented reduction's edge rows [groups][2][m] and flags.
struct SortedWs {
  Radix<uint2> sort;
  float* edge;
  uint32_t* flags;
  int span;
  int64_t groups;
};

// Pairs per group of the segmented reduction: 256, fewer when that would leave
// CUs idle (about 32 groups per CU for 256 CUs).
int seg_span(int64_t n) {
  int64_t span = (n + 256 * 32 - 1) / (256 * 32);
  return (int)(span < SEG_BATCH ? SEG_BATCH : (span > SEG_SPAN ? SEG_SPAN : span));
}

size_t sorted_layout(int64_t L, int32_t m, SortedWs* ws, char* base) {
  Carver c{base};
  const int64_t n = L * NB;
  char* ka = c.take(n * 4);
  char* kb = c.take(n * 4);
  char* va = c.take(n * 8);
  char* vb = c.take(n * 8);
  carve_radix_scratch<uint2>(n, c, ws ? &ws->sort : nullptr);
  const int span = seg_span(n);
  const int64_t groups = (n + span - 1) / span;
  char* edge = c.take((size_t)groups * 2 * m * 4);
  char* flags = c.take((size_t)groups * 4);
  if (ws) {
    ws->sort.ka = (uint32_t*)ka;
    ws->sort.kb = (uint32_t*)kb;
    ws->sort.va = (uint2*)va;
    ws->sort.vb = (uint2*)vb;
    ws->edge = (float*)edge;
    ws->flags = (uint32_t*)flags;
    ws->span = span;
    ws->groups = groups;
  }
  return c.off;
}

// Fills an order: closest-point keys, the stable sort (its result lands in
// sort.ka / sort.va whatever the number of passes), and the merge gate's count.
template <bool TH>
int build_order(const float* q, const Params& P, const OrderWs& o, hipStream_t s) {
  Radix<uint32_t> r = o.sort;
  if (radix_passes(P.N) & 1) {  // start from the other buffers so the result lands in ka / va
    std::swap(r.ka, r.kb);
    std::swap(r.va, r.vb);
  }
  // clear the sort's header (digit counts, failure word, gate partials); the
  // key kernel counts the digits and clears the look-back states
  const int passes = radix_passes(P.N);
  const bool small = r.n < SORT_SMALL_STATES;
  const int64_t state_words = (int64_t)passes * r.states * RADIX * (small ? 1 : 2);
  hipLaunchKernelGGL(k_zero_words, dim3((unsigned)((SORT_HDR_WORDS + THREADS - 1) / THREADS)), dim3(THREADS), 0, s,
                     r.hdr, (int64_t)SORT_HDR_WORDS);
  const int64_t kb = (P.L + THREADS - 1) / THREADS;
  hipLaunchKernelGGL(k_cell_key<TH>, dim3((unsigned)(kb < 1024 ? kb : 1024)), dim3(THREADS), 0, s, q, P, r.ka, passes,
                     r.hdr, reinterpret_cast<uint32_t*>(r.state), state_words);
  if (int rc = launched()) return rc;
  if (int rc = small ? radix_passes_run<uint32_t, true, uint32_t>(r, passes, s)
                     : radix_passes_run<uint32_t, true, uint64_t>(r, passes, s))
    return rc;
  // COUNT_UNROLL positions per thread: one round of loads
  const int64_t cb = (P.L + THREADS * COUNT_UNROLL - 1) / (THREADS * COUNT_UNROLL);
  hipLaunchKernelGGL(k_count_shared, dim3((unsigned)(cb < (1 << 20) ? cb : (1 << 20))), dim3(THREADS), 0, s,
                     (const uint32_t*)o.sort.ka, P.L, r.hdr + SORT_COUNT);
  hipLaunchKernelGGL(k_count_finalize, dim3(1), dim3(WAVE), 0, s, (const uint32_t*)(r.hdr + SORT_COUNT),
                     (const uint32_t*)(r.hdr + SORT_FAIL), o.shared);
  return launched();
}

// q is the lookups' input: q [L][8], or z [L][16] when TH (activation layer).
// The atomic backward kernel for lists of KS; gate is the merged scatter's
// device-side choice (null: always scatter); perm an order to visit the
// lookups in (null: index order); saved the forward's lists (or off).
template <int DT, int M, bool TH, int KS>
void launch_atomic(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                   const uint32_t* gate, const uint32_t* perm, NbrList saved, hipStream_t s) {
  const dim3 grid(grid_for(P)), b(THREADS);
  uint32_t* const nk = nullptr;
  uint2* const nv = nullptr;
  if constexpr (!TH && KS == NB) {
    if (perm && saved.on())
      hipLaunchKernelGGL((k_backward<DT, M, false, false, NB, true, true>), grid, b, 0, s, q, P, table, g, gt, gq, nk,
                         nv, gate, perm, saved);
    else if (perm)
      hipLaunchKernelGGL((k_backward<DT, M, false, false, NB, true, false>), grid, b, 0, s, q, P, table, g, gt, gq,
                         nk, nv, gate, perm, saved);
    else if (saved.on())
      hipLaunchKernelGGL((k_backward<DT, M, false, false, NB, false, true>), grid, b, 0, s, q, P, table, g, gt, gq,
                         nk, nv, gate, perm, saved);
    else
      hipLaunchKernelGGL((k_backward<DT, M, false, false, NB>), grid, b, 0, s, q, P, table, g, gt, gq, nk, nv, gate,
                         perm, saved);
  } else {
    hipLaunchKernelGGL((k_backward<DT, M, false, TH, KS>), grid, b, 0, s, q, P, table, g, gt, gq, nk, nv, gate,
                       perm, saved);
  }
}

// The merged scatter for lists of KS: the lookup order (unless the caller
// passed one: have_order), then both the atomic kernel and the merged kernel --
// the gate's count decides on the device which one works (thinly spread
// queries have nothing to merge and keep the atomic kernel's occupancy).
template <int DT, int M, bool TH, int KS>
int merged_pass(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const OrderWs& o, bool have_order, NbrList saved, hipStream_t s) {
  if (!gt) {
    launch_atomic<DT, M, TH, KS>(q, P, table, g, gt, gq, nullptr, nullptr, saved, s);
    return launched();
  }
  if (!have_order)
    if (int rc = build_order<TH>(q, P, o, s)) return rc;
  launch_atomic<DT, M, TH, KS>(q, P, table, g, gt, gq, o.shared, nullptr, saved, s);
  if (int rc = launched()) return rc;
  // one batch of at most merge_t<KS>() lookups per workgroup
  Params Pm = P;
  Pm.lpw = P.lpw < merge_lpw<KS>() ? P.lpw : merge_lpw<KS>();
  const int64_t per_block = (int64_t)Pm.lpw * WAVES;
  const dim3 grid((unsigned)((P.L + per_block - 1) / per_block));
  const uint32_t* keys = o.sort.ka;
  const uint32_t* perm = o.sort.va;
  if constexpr (!TH && KS == NB) {
    if (saved.on()) {
      hipLaunchKernelGGL((k_backward_merged<DT, M, false, NB, true>), grid, dim3(THREADS), 0, s, q, Pm, table, g, gt,
                         gq, keys, perm, (const uint32_t*)o.shared, saved);
      return launched();
    }
  }
  hipLaunchKernelGGL((k_backward_merged<DT, M, TH, KS>), grid, dim3(THREADS), 0, s, q, Pm, table, g, gt, gq, keys,
                     perm, (const uint32_t*)o.shared, saved);
  return launched();
}

// width: list width (16, 32, 64 or KALL); th: the activation layer (width 32 only).
template <int DT, int M>
struct BwdAtomicLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq, bool th,
                int width, const uint32_t* perm, NbrList saved, hipStream_t s) {
    if (th) {
      launch_atomic<DT, M, true, NB>(q, P, table, g, gt, gq, nullptr, perm, saved, s);
    } else {
      switch (width) {
        case 16: launch_atomic<DT, M, false, 16>(q, P, table, g, gt, gq, nullptr, perm, saved, s); break;
        case 64: launch_atomic<DT, M, false, 64>(q, P, table, g, gt, gq, nullptr, perm, saved, s); break;
        case KALL: launch_atomic<DT, M, false, KALL>(q, P, table, g, gt, gq, nullptr, perm, saved, s); break;
        default: launch_atomic<DT, M, false, NB>(q, P, table, g, gt, gq, nullptr, perm, saved, s); break;
      }
    }
    return launched();
  }
};

template <int DT, int M>
struct BwdMergedLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const OrderWs& o, bool have_order, bool th, int width, NbrList saved, hipStream_t s) {
    if (th) return merged_pass<DT, M, true, NB>(q, P, table, g, gt, gq, o, have_order, saved, s);
    switch (width) {
      case 16: return merged_pass<DT, M, false, 16>(q, P, table, g, gt, gq, o, have_order, saved, s);
      case 64: return merged_pass<DT, M, false, 64>(q, P, table, g, gt, gq, o, have_order, saved, s);
      case KALL: return merged_pass<DT, M, false, KALL>(q, P, table, g, gt, gq, o, have_order, saved, s);
      default: return merged_pass<DT, M, false, NB>(q, P, table, g, gt, gq, o, have_order, saved, s);
    }
  }
};

template <int DT, int M>
struct BwdSortedLaunch {
  static int go(const float* q, const Params& P, const void* table, const float* g, float* gt, float* gq,
                const SortedWs& ws, bool th, NbrList saved, hipStream_t s) {
    const dim3 grid(grid_for(P)), b(THREADS);
    const uint32_t* const np = nullptr;
    if (th)
      hipLaunchKernelGGL((k_backward<DT, M, true, true>), grid, b, 0, s, q, P, table, g, gt, gq, ws.sort.ka,
                         ws.sort.va, np, np, saved);
    else if (saved.on())
      hipLaunchKernelGGL((k_backward<DT, M, true, false, NB, false, true>), grid, b, 0, s, q, P, table, g, gt, gq,
                         ws.sort.ka, ws.sort.va, np, np, saved);
    else
      hipLaunchKernelGGL((k_backward<DT, M, true, false>), grid, b, 0, s, q, P, table, g, gt, gq, ws.sort.ka,
                         ws.sort.va, np, np, saved);
    int rc = launched();
    if (rc || !gt) return rc;
    if ((rc = radix_sort<uint2, false>(ws.sort, P.N, s))) return rc;  // keys lie in [0, N]
    const bool odd = radix_passes(P.N) & 1;
    const uint32_t* keys = odd ? ws.sort.kb : ws.sort.ka;
    const uint2* vals = odd ? ws.sort.vb : ws.sort.va;
    const int64_t per_block = THREADS / M;
    const unsigned blocks = (unsigned)((ws.groups + per_block - 1) / per_block);
    hipLaunchKernelGGL((k_segreduce<M>), dim3(blocks), b, 0, s, keys, vals, ws.sort.n, P.N, (uint32_t)P.L, g, gt,
                       ws.span, ws.edge,
                       ws.flags);
    hipLaunchKernelGGL((k_segfix<M>), dim3(blocks), b, 0, s, keys, ws.sort.n, ws.span, (const float*)ws.edge,
                       (const uint32_t*)ws.flags, ws.groups, gt);
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
      default:
        hipLaunchKernelGGL((k_forward<DT, M, false>), g, b, 0, s, q, P, table, out, (const uint32_t*)nullptr,
                           NbrList{nullptr, nullptr, nullptr});
        break;
    }
    return launched();
  }
};

// An order passed by the caller: 256-byte aligned and large enough for L
// lookups; its positions (perm) then address the lookups.
int check_order(const void* order, size_t bytes, int64_t L, OrderWs* o) {
  if (!order) return LRAM_OK;
  if ((reinterpret_cast<uintptr_t>(order) & 255) || bytes < order_layout(L, nullptr, nullptr)) return LRAM_EINVAL;
  order_layout(L, o, reinterpret_cast<char*>(const_cast<void*>(order)));
  return LRAM_OK;
}

// Saved lists: all three arrays or none, 4-byte aligned.
int check_saved(const void* slot, const void* w, const void* code, NbrList* nl) {
  const int given = (slot != nullptr) + (w != nullptr) + (code != nullptr);
  if (given != 0 && given != 3) return LRAM_EINVAL;
  if (misaligned4(slot) || misaligned4(w) || misaligned4(code)) return LRAM_EINVAL;
  *nl = NbrList{(int32_t*)slot, (float*)w, (uint32_t*)code};
  return LRAM_OK;
}

int forward_impl(const float* in, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype, int64_t N,
                 int32_t m, void* out, const void* order, size_t order_bytes, NbrList save, bool th,
                 hipStream_t stream) {
  int64_t L;
  Params P;
  int rc = check_common(in, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  OrderWs o{};
  if ((rc = check_order(order, order_bytes, L, &o))) return rc;
  if (L == 0) return LRAM_OK;
  if (!out || misaligned16(out)) return LRAM_EINVAL;
  return dispatch<FwdLaunch>(dtype, m, in, P, table, out, th, order ? (const uint32_t*)o.sort.va : nullptr, save,
                             stream);
}

int resolve_mode(int64_t B, int64_t H, int mode, int* resolved);

// width: list width (NB for lram_backward and the activation layer).
int backward_impl(const float* in, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_in, const void* order,
                  size_t order_bytes, NbrList saved, int mode, void* workspace, size_t ws_bytes, int width, bool th,
                  hipStream_t stream) {
  int64_t L;
  Params P;
  int rc = check_common(in, B, H, K, &L, &P);
  if (rc) return rc;
  rc = check_table(table, dtype, N, m, P, L);
  if (rc) return rc;
  if ((rc = resolve_mode(B, H, mode, &mode))) return rc;
  if (mode == LRAM_SCATTER_SORTED && width != NB) return LRAM_EMODE;  // the sorted scatter takes k = 32
  OrderWs o{};
  if ((rc = check_order(order, order_bytes, L, &o))) return rc;
  if (L == 0) return LRAM_OK;
  if (!grad_out || misaligned16(grad_out)) return LRAM_EINVAL;
  if (!grad_table && !grad_in) return LRAM_EINVAL;
  if (grad_table && misaligned16(grad_table)) return LRAM_EINVAL;
  if (grad_in && misaligned16(grad_in)) return LRAM_EINVAL;
  if (mode == LRAM_SCATTER_ATOMIC)
    return dispatch<BwdAtomicLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, th, width,
                                     order ? (const uint32_t*)o.sort.va : nullptr, saved, stream);
  if (mode == LRAM_SCATTER_MERGED) {
    if (!order) {
      const size_t need = order_layout(L, nullptr, nullptr);
      if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LRAM_EWORKSPACE;
      order_layout(L, &o, reinterpret_cast<char*>(workspace));
    }
    return dispatch<BwdMergedLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, o, order != nullptr, th,
                                     width, saved, stream);
  }
  if (L * NB >= (int64_t(1) << 32)) return LRAM_EINVAL;  // the sorted scatter's pair positions are 32-bit
  const size_t need = sorted_layout(L, m, nullptr, nullptr);
  if (!workspace || ws_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LRAM_EWORKSPACE;
  SortedWs ws;
  sorted_layout(L, m, &ws, reinterpret_cast<char*>(workspace));
  return dispatch<BwdSortedLaunch>(dtype, m, in, P, table, grad_out, grad_table, grad_in, ws, th, saved, stream);
}

int resolve_mode(int64_t B, int64_t H, int mode, int* resolved) {
  if (!resolved || B < 0 || H < 0 || (H != 0 && B > INT64_MAX / H)) return LRAM_EINVAL;
  if (mode < LRAM_SCATTER_ATOMIC || mode > LRAM_SCATTER_AUTO) return LRAM_EMODE;
  *resolved = mode != LRAM_SCATTER_AUTO ? mode : (B * H >= AUTO_MERGE_MIN ? LRAM_SCATTER_MERGED : LRAM_SCATTER_ATOMIC);
  return LRAM_OK;
}

constexpr NbrList NO_LIST{nullptr, nullptr, nullptr};

// Workspace of lram_backward_noalloc: one copy per GPU, held from the code
// object's load until the process ends.  Host code never uses the name as an
// address (it stands for a host-side shadow): scratch_address() fetches each
// device's own address once with hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[LRAM_STATIC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device (null and LRAM_EHIP on failure).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    g_last_hip_error = (int)e;
    return LRAM_EHIP;
  }
  if (dev < 0 || dev >= MAX_DEVICES) return LRAM_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      g_last_hip_error = (int)e;
      return LRAM_EHIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return LRAM_OK;
}

}  // namespace

extern "C" {

int lram_version(void) { return 200; }

const char* lram_strerror(int status) {
  switch (status) {
    case LRAM_OK: return "ok";
    case LRAM_EINVAL: return "invalid argument (null/misaligned pointer, negative size or undersized buffer)";
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
  if (!slot || !w || misaligned4(slot) || misaligned4(w) || misaligned4(d2)) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_neighbors<NB>, dim3(grid_for(P)), dim3(THREADS), 0, (hipStream_t)stream, q, P, slot, w, d2);
  return launched();
}

int lram_order_bytes(int64_t B, int64_t H, size_t* bytes, size_t* keys_offset, size_t* perm_offset) {
  if (!bytes || B < 0 || H < 0 || (H != 0 && B > INT64_MAX / H) || B * H > LMAX) return LRAM_EINVAL;
  const int64_t L = B * H;
  *bytes = order_layout(L, nullptr, nullptr);
  if (keys_offset) *keys_offset = ORDER_KEYS_OFFSET;
  if (perm_offset) *perm_offset = ORDER_KEYS_OFFSET + align256((size_t)L * 4);
  return LRAM_OK;
}

int lram_order(const float* q, int64_t B, int64_t H, const int32_t K[8], void* order, size_t order_bytes,
               void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (!order) return LRAM_EINVAL;
  OrderWs o;
  if ((rc = check_order(order, order_bytes, L, &o))) return rc;
  if (L == 0) return LRAM_OK;
  return build_order<false>(q, P, o, (hipStream_t)stream);
}

int lram_forward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                 int64_t N, int32_t m, void* out, const void* order, size_t order_bytes, int32_t* nbr_slot,
                 float* nbr_w, uint32_t* nbr_code, void* stream) {
  NbrList nl;
  if (int rc = check_saved(nbr_slot, nbr_w, nbr_code, &nl)) return rc;
  return forward_impl(q, B, H, K, table, dtype, N, m, out, order, order_bytes, nl, false, (hipStream_t)stream);
}

int lram_theta_forward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                       int64_t N, int32_t m, void* out, void* stream) {
  return forward_impl(z, B, H, K, table, dtype, N, m, out, nullptr, 0, NO_LIST, true, (hipStream_t)stream);
}

int lram_theta_coords(const float* z, int64_t B, int64_t H, const int32_t K[8], float* q, float* s, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(z, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!q || misaligned16(q) || misaligned4(s)) return LRAM_EINVAL;
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
  if (H != 0 && B > INT64_MAX / H / NB) return LRAM_EINVAL;
  *bytes = mode == LRAM_SCATTER_SORTED ? sorted_layout(B * H, m, nullptr, nullptr)
                                       : order_layout(B * H, nullptr, nullptr);
  return LRAM_OK;
}

int lram_backward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, const void* order,
                  size_t order_bytes, const int32_t* nbr_slot, const float* nbr_w, const uint32_t* nbr_code, int mode,
                  void* workspace, size_t ws_bytes, void* stream) {
  NbrList nl;
  if (int rc = check_saved(nbr_slot, nbr_w, nbr_code, &nl)) return rc;
  return backward_impl(q, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_q, order, order_bytes, nl, mode,
                       workspace, ws_bytes, NB, false, (hipStream_t)stream);
}

int lram_backward_noalloc(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                          int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, int mode,
                          void* stream) {
  size_t need = 0;
  if (int rc = lram_backward_workspace_bytes(B, H, m, mode, &need)) return rc;
  if (need > LRAM_STATIC_SCRATCH_BYTES) return LRAM_EWORKSPACE;
  void* ws = nullptr;
  if (need > 0)
    if (int rc = scratch_address(&ws)) return rc;
  return backward_impl(q, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_q, nullptr, 0, NO_LIST, mode, ws,
                       need > 0 ? LRAM_STATIC_SCRATCH_BYTES : 0, NB, false, (hipStream_t)stream);
}

int lram_theta_backward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                        int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_z, int mode,
                        void* workspace, size_t ws_bytes, void* stream) {
  return backward_impl(z, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_z, nullptr, 0, NO_LIST, mode,
                       workspace, ws_bytes, NB, true, (hipStream_t)stream);
}
int lram_access_histogram(const float* q, int64_t B, int64_t H, const int32_t K[8], float* hist, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!hist || misaligned4(hist)) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_access_hist, dim3(grid_for(P)), dim3(THREADS), 0, (hipStream_t)stream, q, P, hist);
  return launched();
}

int lram_access_stats(const float* hist, int64_t N, double* out, void* stream) {
  if (N <= 0 || !hist || !out || misaligned4(hist) || (reinterpret_cast<uintptr_t>(out) & 7)) return LRAM_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(k_fill_f64, dim3(1), dim3(WAVE), 0, s, out, 4, 0.0);
  const int64_t blocks = (N + THREADS - 1) / THREADS;
  hipLaunchKernelGGL(k_access_reduce, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(THREADS), 0, s, hist,
                     N, out);
  hipLaunchKernelGGL(k_access_finalize, dim3(1), dim3(WAVE), 0, s, out, N);
  return launched();
}

// Checks of the Adam entry points and their step constants (1 - beta and the
// bias corrections formed in fp64, rounded once).
static int adam_args(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg, float* exp_avg_sq,
                     int64_t step, double lr, double beta1, double beta2, double eps, AdamArgs* a) {
  if (dtype != LRAM_F32 && dtype != LRAM_BF16) return LRAM_EDTYPE;
  if (m != 32 && m != 64) return LRAM_EDTYPE;
  if (N < 0 || step < 1 || !(lr >= 0.0) || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) ||
      !(eps >= 0.0))
    return LRAM_EINVAL;
  if (N == 0) return LRAM_OK;
  for (const void* ptr : {(const void*)table, (const void*)grad, (const void*)exp_avg, (const void*)exp_avg_sq})
    if (!ptr || misaligned16(ptr)) return LRAM_EINVAL;
  a->lr = (float)lr;
  a->beta1 = (float)beta1;
  a->beta2 = (float)beta2;
  a->eps = (float)eps;
  a->om1 = (float)(1.0 - beta1);
  a->om2 = (float)(1.0 - beta2);
  a->bc1 = (float)(1.0 - std::pow(beta1, (double)step));
  a->bc2 = (float)(1.0 - std::pow(beta2, (double)step));
  return LRAM_OK;
}

int lram_sparse_adam(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg, float* exp_avg_sq,
                     int64_t step, double lr, double beta1, double beta2, double eps, void* stream) {
  AdamArgs a;
  if (int rc = adam_args(table, dtype, N, m, grad, exp_avg, exp_avg_sq, step, lr, beta1, beta2, eps, &a)) return rc;
  if (N == 0) return LRAM_OK;
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

int lram_mark_touched(const float* q, int64_t B, int64_t H, const int32_t K[8], uint8_t* touched, void* stream) {
  int64_t L;
  Params P;
  int rc = check_common(q, B, H, K, &L, &P);
  if (rc) return rc;
  if (L == 0) return LRAM_OK;
  if (!touched) return LRAM_EINVAL;
  hipLaunchKernelGGL(k_mark_touched, dim3(grid_for(P)), dim3(THREADS), 0, (hipStream_t)stream, q, P, touched);
  return launched();
}

int lram_sparse_adam_touched(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg,
                             float* exp_avg_sq, uint8_t* touched, int64_t step, double lr, double beta1, double beta2,
                             double eps, void* stream) {
  AdamArgs a;
  if (int rc = adam_args(table, dtype, N, m, grad, exp_avg, exp_avg_sq, step, lr, beta1, beta2, eps, &a)) return rc;
  if (N == 0) return LRAM_OK;
  if (!touched) return LRAM_EINVAL;
  const int64_t rows_per_block = (int64_t)WAVES * WAVE;
  int64_t blocks = (N + rows_per_block - 1) / rows_per_block;
  blocks = blocks < 16384 ? blocks : 16384;
  const dim3 g((unsigned)blocks), b(THREADS);
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LRAM_F32 && m == 32) hipLaunchKernelGGL((k_sparse_adam_touched<LRAM_F32, 32>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, touched, a);
  if (dtype == LRAM_F32 && m == 64) hipLaunchKernelGGL((k_sparse_adam_touched<LRAM_F32, 64>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, touched, a);
  if (dtype == LRAM_BF16 && m == 32) hipLaunchKernelGGL((k_sparse_adam_touched<LRAM_BF16, 32>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, touched, a);
  if (dtype == LRAM_BF16 && m == 64) hipLaunchKernelGGL((k_sparse_adam_touched<LRAM_BF16, 64>), g, b, 0, s, table, N, grad, exp_avg, exp_avg_sq, touched, a);
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
  if (!slot || !w || misaligned4(slot) || misaligned4(w) || misaligned4(d2)) return LRAM_EINVAL;
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
  if (!out || misaligned16(out)) return LRAM_EINVAL;
  return dispatch<FwdKLaunch>(dtype, m, q, P, table, out, width, (hipStream_t)stream);
}

int lram_backward_k(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                    int64_t N, int32_t m, int32_t k, const float* grad_out, float* grad_table, float* grad_q,
                    int mode, void* workspace, size_t ws_bytes, void* stream) {
  const int width = list_width(k);
  if (!width) return LRAM_EINVAL;
  return backward_impl(q, B, H, K, table, dtype, N, m, grad_out, grad_table, grad_q, nullptr, 0, NO_LIST, mode,
                       workspace, ws_bytes,
                       width, false, (hipStream_t)stream);
}

}  // extern "C"
