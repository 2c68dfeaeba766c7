/*
 * lram.h -- C ABI of liblram.so, the LRAM lattice lookup on AMD Instinct MI355X (gfx950).
 *
 * Goucher & Troll, "Differentiable Random Access Memory using Lattices":
 * a memory of N = prod K_i value vectors v_s in R^m stored at the locations of
 * the lattice Lambda = 2*E8 (Sec. 2.4) on the torus T_K (Sec. 2.2).  A lookup
 * maps a query q in R^8 to
 *
 *     phi(q) = sum_{j < 32} f(|x - k_j|) v_{slot(k_j)},   f(r) = max(0, 1 - r^2/8)^4,
 *
 * over the 32 lattice points k_j closest to x (Sec. 2.5 kernel, Sec. 2.6
 * truncation to k = 32, no renormalisation).
 *
 * Conventions shared by every entry point:
 *   - Scale.  q is given at the unimodular-E8 scale on a torus of side K_i, so
 *     q_i in [0, K_i) covers it once; the lattice work happens at the doubled
 *     scale of Sec. 2.4, x_i = fmodf(2 q_i, 2 K_i) (exact; a negative q_i keeps
 *     its sign; any real q_i is accepted).
 *   - K.  Eight even integers 2 <= K_i <= 8192 (host array); N = prod K_i < 2^31.
 *     (8192 keeps every lattice coordinate of the doubled scale inside int16;
 *     with N < 2^31 it only excludes tori that are nearly one-dimensional.)
 *   - Locations.  slot(k) = eps*N/2 + ((..(Y_0 K_1 + Y_1) K_2 + ..) K_6 + Y_6)*(K_7/2)
 *     + floor(Y_7/2), with eps = k_0 mod 2 and Y_i = ((k_i - eps)/2) mod K_i:
 *     row slot of the value table holds v at that location (Sec. 2.2, M = Lambda/L_K).
 *   - Selection.  The squared distance that decides the 32 is the fp32 recipe
 *     e_i = fl(x_i - k_i), s = e_0^2, s = fl(s + fl(e_i^2)) for i = 1..7, no
 *     FMA; support is s < 8 (open ball, Sec. 2.5); order is ascending
 *     (bits of s, slot, k lexicographic).  Fewer than 32 points in the support
 *     (only at exceptional queries such as lattice points or deep holes) are
 *     padded with slot -1 and weight 0.  A non-finite query coordinate gives an
 *     all-padding list.
 *   - Layout.  Every tensor is dense row-major: q [L][8] fp32, table [N][m],
 *     out [L][m] (table dtype), grad_out [L][m] fp32, grad_table [N][m] fp32,
 *     grad_q [L][8] fp32, with L = B*H < 2^31 lookups (heads share the
 *     table, Sec. 2.3).  Device pointers must be 16-byte aligned, except the
 *     per-element outputs slot, w, d2, s and hist, which need 4 bytes.
 *   - dtype/m.  LRAM_F32 or LRAM_BF16 tables with m in {32, 64}; accumulation is
 *     always fp32.
 *   - Streams.  stream is a hipStream_t (NULL = the null stream).  All work is
 *     enqueued asynchronously; nothing synchronises.  Arguments are checked on
 *     the host before anything is launched; a failed check launches nothing.
 *   - Memory.  The caller owns every buffer.  The library allocates no device
 *     memory and keeps no mutable global state: calls on different streams
 *     may overlap (but see lram_backward on grad_table).
 *   - Errors.  Return value LRAM_OK (0) or one of lram_status below.  Faults of
 *     the asynchronous kernels surface at the caller's next synchronisation.
 */
#ifndef LRAM_H
#define LRAM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LRAM_NEIGHBOURS 32
#define LRAM_ALL 0            /* k of the untruncated lookup: every point of the support */
#define LRAM_MAX_SUPPORT 256  /* list width of the untruncated lookup */

typedef enum {
  LRAM_OK = 0,
  LRAM_EINVAL = 1,      /* null pointer with L > 0, negative size, L >= 2^31, misaligned pointer,
                           undersized order buffer, saved lists incomplete */
  LRAM_EBADK = 2,       /* a K_i odd, < 2 or > 8192, N != prod K, or N >= 2^31 */
  LRAM_EDTYPE = 3,      /* unknown dtype or unsupported m for that dtype */
  LRAM_EWORKSPACE = 4,  /* workspace missing or smaller than lram_backward_workspace_bytes */
  LRAM_EMODE = 5,       /* unknown scatter mode, or the sorted mode with k != 32 */
  LRAM_EHIP = 6         /* a HIP launch failed; see lram_last_hip_error */
} lram_status;

typedef enum { LRAM_F32 = 0, LRAM_BF16 = 1 } lram_dtype;

typedef enum {
  LRAM_SCATTER_ATOMIC = 0, /* fp32 atomic adds straight into grad_table */
  LRAM_SCATTER_SORTED = 1, /* sort (slot, lookup) pairs, one read-modify-write per touched row;
                              bit-reproducible from call to call */
  LRAM_SCATTER_MERGED = 2, /* order lookups by their closest lattice point, merge equal slots within
                              each batch of consecutive lookups (64 for lists of up to 32, 32 for
                              longer ones), one atomic row per distinct slot;
                              when fewer than a tenth of the lookups share their closest point with
                              another (nothing to merge) the device falls back to the atomic scatter */
  LRAM_SCATTER_AUTO = 3    /* MERGED for L >= 131072 lookups, ATOMIC below (the sort does not pay off) */
} lram_scatter_mode;

/* Library version (major*10000 + minor*100 + patch): 200 = 0.2.0. */
int lram_version(void);

/* Static description of a status code. */
const char* lram_strerror(int status);

/* hipError_t of the most recent LRAM_EHIP on the calling thread (0 if none). */
int lram_last_hip_error(void);

/*
 * lram_neighbors -- the neighbour lists themselves (Sec. 2.6: the kernel's
 * indices alpha_i and weights w_i).  For each of L = B*H lookups writes, in
 * selection order:
 *   slot [L][32] int32  locations, -1 for padding
 *   w    [L][32] fp32   fp32 recipe weight u = fl(1 - s*0.125f), w = fl(fl(u*u)*fl(u*u)); 0 for padding
 *   d2   [L][32] fp32   recipe squared distance s (nullable); +inf for padding
 * Device pointers.  B, H >= 0; B*H == 0 is a no-op.
 */
int lram_neighbors(const float* q, int64_t B, int64_t H, const int32_t K[8], int32_t* slot, float* w,
                   float* d2, void* stream);

/*
 * Lookup order (Sec. 2.6: lookups whose queries share their closest lattice
 * point share most of their 32 neighbours).
 *
 * lram_order_bytes -- size of an order buffer for L = B*H lookups (host only),
 * and the byte offsets of its two documented arrays (nullable outputs).
 *
 * lram_order -- fills `order` (device, 256-byte aligned, at least
 * lram_order_bytes) for the queries q: the lookups sorted, stably, by the
 * location of their closest lattice point (the first point of Sec. 2.6's
 * reduction; where several points are equally close in exact arithmetic, one
 * of them -- not necessarily the one the fp32 distance recipe lists first):
 *   bytes [0, 4)            uint32: how many lookups share their key with a
 *                           neighbour in the order (decides, on the device,
 *                           whether the merged scatter merges)
 *   bytes [4, 8)            uint32: 0; nonzero if a workgroup of the sort gave
 *                           up waiting for its predecessors' digit counts (never
 *                           expected; the order is then not sorted, though every
 *                           position still names a lookup below L or is skipped)
 *   keys  [L] uint32        at keys_offset: the sorted keys (location, or N for a
 *                           non-finite query)
 *   perm  [L] uint32        at perm_offset: the lookup at each position
 *   the rest                scratch of the sort.
 * The same buffer serves as the merged scatter's workspace.  An order may be
 * passed to lram_forward and lram_backward of the same q, B, H and K: both then
 * visit the lookups in this order (workgroups take consecutive positions, each
 * XCD one contiguous range, so lookups that read the same rows run on the
 * same L2), and the merged scatter uses it instead of sorting again.  An order
 * written for other queries gives wrong results but never addresses outside
 * the caller's buffers (positions outside [0, L) are skipped).
 */
int lram_order_bytes(int64_t B, int64_t H, size_t* bytes, size_t* keys_offset, size_t* perm_offset);
int lram_order(const float* q, int64_t B, int64_t H, const int32_t K[8], void* order, size_t order_bytes,
               void* stream);

/*
 * lram_forward -- out[l][:] = sum_j w_j table[slot_j][:] (Sec. 2.2 with the
 * truncation of Sec. 2.6), fp32 accumulation, written once in the table dtype
 * (bf16: round to nearest even).  table holds N rows of m elements.
 *   order/order_bytes  nullable: an order from lram_order for these queries
 *                      (the lookups are then visited in that order; out is the
 *                      same).
 *   nbr_slot [L][32] int32, nbr_w [L][32] fp32, nbr_code [L][32] uint32:
 *                      nullable (all three or none): the neighbour lists saved
 *                      for lram_backward (Sec. 2.6: the kernel hands the
 *                      indices alpha_i and the weights w_i to the autograd
 *                      wrapper).  Entry j of lookup l: the location (-1 for
 *                      padding), the recipe weight, and the point's coordinates
 *                      p in its query's fundamental-region frame (Sec. 2.6:
 *                      the point is c + sigma pi^-1 p for the query's closest
 *                      point c and signed permutation sigma pi), eight 3-bit
 *                      fields p_r + 3 in bits [3r, 3r + 3), 0 for padding.  The
 *                      32 entries are those of lram_neighbors in the search's
 *                      own order (padding last).  384 bytes per lookup.
 */
int lram_forward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                 int64_t N, int32_t m, void* out, const void* order, size_t order_bytes, int32_t* nbr_slot,
                 float* nbr_w, uint32_t* nbr_code, void* stream);

/*
 * lram_backward_workspace_bytes -- device workspace needed by lram_backward
 * (and lram_backward_k, lram_theta_backward) for L = B*H lookups in the given
 * scatter mode (0 for LRAM_SCATTER_ATOMIC; the same for every k; the merged
 * scatter's workspace is an order buffer, lram_order_bytes).
 */
int lram_backward_workspace_bytes(int64_t B, int64_t H, int32_t m, int mode, size_t* bytes);

/*
 * lram_scatter_mode_resolved -- the concrete mode (ATOMIC, SORTED or MERGED)
 * that lram_backward runs for L = B*H lookups when given `mode` (host only).
 */
int lram_scatter_mode_resolved(int64_t B, int64_t H, int mode, int* resolved);

/*
 * lram_backward -- gradients of sum_l <grad_out[l], phi(q_l)> with the selection
 * held fixed (Sec. 2.6: the kernel supplies the weights and their derivatives
 * to an autograd wrapper):
 *   grad_table[s][:] += sum over (l, j) with slot_j(l) = s of w_j grad_out[l][:]
 *       (accumulated: the caller zeroes grad_table once; untouched rows are not
 *        written; concurrent calls on other streams that update the same
 *        grad_table race only in rounding order under LRAM_SCATTER_ATOMIC and
 *        LRAM_SCATTER_MERGED, whose row adds are atomic, and must not overlap
 *        under LRAM_SCATTER_SORTED)
 *   grad_q[l][i] = sum_j -2 u_j^3 (x_i - k_{j,i}) <grad_out[l], table[slot_j]>,
 *       u_j = 1 - s_j/8 (overwritten; nullable to skip it)
 * order/order_bytes: nullable; an order from lram_order for these queries.
 * The merged scatter then takes it instead of sorting (no workspace needed),
 * the atomic one visits the lookups in it, the sorted one ignores it.
 * nbr_slot/nbr_w/nbr_code: nullable (all three or none); the lists lram_forward
 * saved for these queries replace the neighbour search (each entry's distance
 * is recomputed from its code for dq).  Entries whose location is outside
 * [0, N) count as padding, so lists of other queries give wrong gradients but
 * never address outside grad_table.  Without them the search is recomputed
 * from q.
 * workspace/ws_bytes: device buffer, 256-byte aligned, of at least
 * lram_backward_workspace_bytes (may be NULL for the atomic mode, and for the
 * merged mode when an order is given); its contents on entry do not matter,
 * and calls that may overlap need workspaces of their own.
 * LRAM_SCATTER_SORTED is bit-reproducible: the same inputs give the same
 * grad_table bits on every call (every row's sum is formed in one fixed
 * order, each row written by one thread group); it needs 32 L < 2^32.  The
 * atomic and merged modes add in an order that varies from call to call.
 * grad_table may be NULL only if grad_q is not (without grad_table every mode
 * computes grad_q the same way, bit for bit).
 */
int lram_backward(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                  int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, const void* order,
                  size_t order_bytes, const int32_t* nbr_slot, const float* nbr_w, const uint32_t* nbr_code,
                  int mode, void* workspace, size_t ws_bytes, void* stream);

/*
 * lram_backward_noalloc -- lram_backward (no order, no saved lists) for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  The workspace of the
 * sorted and merged scatters is a static array inside the library, one per
 * GPU, LRAM_STATIC_SCRATCH_BYTES long, held from the library's first use on a
 * GPU until the process ends; the call itself allocates nothing.  Up to
 * 4.6 M lookups fit the merged scatter's order (the billion-location
 * workload's 4,194,304 included), about 100 K the sorted scatter's pairs;
 * larger calls return LRAM_EWORKSPACE (the atomic mode needs no workspace and
 * takes any size).  Every call on a GPU shares that GPU's array: calls that
 * may overlap on one GPU (other streams, other host threads) race on it and
 * must not be issued.  The stream must belong to the current device.
 */
#define LRAM_STATIC_SCRATCH_BYTES ((size_t)80 << 20)
int lram_backward_noalloc(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                          int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_q, int mode,
                          void* stream);

/*
 * Training-side companions.
 *
 * lram_access_histogram -- hist[s] += sum of the kernel weights w_j of the
 * (lookup, neighbour) pairs whose location is s (the weighted accesses of the
 * utilisation table, Sec. 4.3); hist [N] fp32 device, accumulated (fp32 atomics).
 *
 * lram_access_stats -- from hist [N]: out (device, 4 doubles, 8-byte aligned,
 * overwritten) = {fraction of locations with hist > 0, KL divergence of the
 * distribution hist / sum(hist) from uniform (nats), sum(hist), number of
 * locations with hist > 0}.  fp64 reductions.
 *
 * lram_sparse_adam -- one Adam step (Sec. 3.2 trains the memory with Adam,
 * learning rate 1e-3; Algorithm 1 of Adam: m = b1 m + (1-b1) g,
 * v = b2 v + (1-b2) g^2, table -= lr (m / (1-b1^step)) / (sqrt(v / (1-b2^step)) + eps))
 * on the rows whose gradient row in grad [N][m] fp32 is not identically zero;
 * other rows keep value and moments (the lazy, sparse form).  exp_avg and
 * exp_avg_sq are [N][m] fp32 (zero-initialised by the caller), table is
 * [N][m] in dtype (bf16: updated in fp32, rounded once).  grad rows that were
 * used are cleared to zero.  step >= 1; lr, beta1, beta2, eps are host
 * doubles: 1 - beta and the bias corrections 1 - beta^step are formed in fp64
 * and rounded once (beta2 = 0.999 in fp32 would move 1 - beta2^step by
 * 1e-5 relative); the per-entry arithmetic is fp32.
 */
int lram_access_histogram(const float* q, int64_t B, int64_t H, const int32_t K[8], float* hist, void* stream);
int lram_access_stats(const float* hist, int64_t N, double* out, void* stream);
int lram_sparse_adam(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg, float* exp_avg_sq,
                     int64_t step, double lr, double beta1, double beta2, double eps, void* stream);

/*
 * lram_mark_touched -- touched[s] = 1 (uint8 [N], device) for every location s
 * in the closest-32 list of every lookup of q (Sec. 2.6): the rows that
 * lram_backward of these lookups writes.  Other entries are left as they are
 * (the caller clears the array once; lram_sparse_adam_touched clears what it
 * uses).
 *
 * lram_sparse_adam_touched -- lram_sparse_adam on the rows whose touched flag
 * is set, in the same arithmetic (a flagged row whose gradient row is
 * identically zero keeps value and moments); the flags of [0, N) are cleared.
 * The step reads the N flag bytes and the flagged rows only, so its cost
 * follows the touched rows rather than the table size (Sec. 3.2: the memory's
 * rows are a sparse parameter; most of a large table is untouched by a step).
 */
int lram_mark_touched(const float* q, int64_t B, int64_t H, const int32_t K[8], uint8_t* touched, void* stream);
int lram_sparse_adam_touched(void* table, int dtype, int64_t N, int32_t m, float* grad, float* exp_avg,
                             float* exp_avg_sq, uint8_t* touched, int64_t step, double lr, double beta1, double beta2,
                             double eps, void* stream);

/*
 * Variable k and the untruncated lookup (Sec. 2.2 and 2.5: the sum over every
 * lattice point in the support; Sec. 2.6: the truncation to the closest k,
 * whose k = 32 is what every other entry point uses).  k is 16, 32, 64 or
 * LRAM_ALL; otherwise LRAM_EINVAL.  The selection is the closest min(k, count)
 * points in the order of the conventions above; LRAM_ALL keeps every point
 * whose recipe distance is below 8.  That is at most 121 points in exact
 * arithmetic (Table 1); the recipe's rounding can admit points at distance
 * exactly sqrt 8, but never more than the 1 + 240 that a ball of that radius
 * holds, so LRAM_ALL lists are LRAM_MAX_SUPPORT wide.  Lists are padded with
 * slot -1, weight 0.  The backward takes the atomic and merged scatters (and
 * LRAM_SCATTER_AUTO); the sorted scatter takes k = 32 only (LRAM_EMODE).
 */

/* lram_neighbors_k -- as lram_neighbors with lists of width w = k (LRAM_MAX_SUPPORT
 * for LRAM_ALL): slot/w/d2 are [L][w]. */
int lram_neighbors_k(const float* q, int64_t B, int64_t H, const int32_t K[8], int32_t k, int32_t* slot, float* w,
                     float* d2, void* stream);

/* lram_forward_k -- out[l] = sum over the closest min(k, count) points of w_j table[slot_j]. */
int lram_forward_k(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                   int64_t N, int32_t m, int32_t k, void* out, void* stream);

/* lram_backward_k -- lram_backward's gradients for the k-point lookup; mode,
 * workspace and ws_bytes as for lram_backward (the merged scatter merges the
 * k pairs of every lookup; a batch holds 64 lookups for k <= 32, 2048/k above). */
int lram_backward_k(const float* q, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                    int64_t N, int32_t m, int32_t k, const float* grad_out, float* grad_table, float* grad_q,
                    int mode, void* workspace, size_t ws_bytes, void* stream);

/*
 * Activation layer in front of the lookup (Sec. 2.3).  Each lookup takes 8
 * complex numbers z_i = z[l][2i] + i z[l][2i+1] (z is [L][16] fp32, 16-byte
 * aligned) and computes
 *
 *     theta(z) = (sum_i 1/|z_i|)^-1 phi(q),   q_i = (K_i / 2 pi) arg z_i,
 *
 * the scale being the displayed formula of Sec. 2.3 (the text calls it a
 * harmonic mean; the formula has no factor 8), so theta(lambda z) =
 * lambda theta(z) for lambda >= 0.  q_i is formed in fp64 (atan2 of the fp32
 * inputs times K_i / 2 pi) and rounded once to fp32; the lookup then proceeds
 * exactly as lram_forward on that q.  A zero z_i gives scale 0 (output 0,
 * gradients 0: the continuous extension); a non-finite input gives output 0
 * and zero gradients.
 */

/* lram_theta_coords -- q [L][8] fp32 and scale s [L] fp32 (nullable) as the
 * activation layer computes them (parity surface). */
int lram_theta_coords(const float* z, int64_t B, int64_t H, const int32_t K[8], float* q, float* s, void* stream);

/* lram_theta_forward -- out[l] = theta(z_l) in the table dtype (fp32
 * accumulation, the scale folded into the 32 weights, one rounding). */
int lram_theta_forward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                       int64_t N, int32_t m, void* out, void* stream);

/*
 * lram_theta_backward -- gradients of sum_l <grad_out[l], theta(z_l)>, selection
 * held fixed:
 *   grad_table[s] += sum over (l, j) with slot_j(l) = s of scale_l w_j grad_out[l]
 *       (accumulated; same modes, workspace and rules as lram_backward, whose
 *        lram_backward_workspace_bytes applies unchanged)
 *   grad_z[l] [16] fp32 (overwritten; nullable): with r_i = |z_i|, c_i = K_i/2pi,
 *       dL/ds = sum_j w_j <G, v_j>, dL/dq = s dq (dq as in lram_backward),
 *       dL/dRe z_i = dL/ds s^2 Re z_i / r_i^3 - dL/dq_i c_i Im z_i / r_i^2,
 *       dL/dIm z_i = dL/ds s^2 Im z_i / r_i^3 + dL/dq_i c_i Re z_i / r_i^2.
 */
int lram_theta_backward(const float* z, int64_t B, int64_t H, const int32_t K[8], const void* table, int dtype,
                        int64_t N, int32_t m, const float* grad_out, float* grad_table, float* grad_z, int mode,
                        void* workspace, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LRAM_H */
