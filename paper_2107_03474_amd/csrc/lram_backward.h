// lram_backward.h -- part of liblram (included by lram.hip only).
//
// Backward: the value-gradient atomic scatter, the query gradient (and the
// activation layer's chain), and the backward kernel of the atomic and sorted
// scatters.

#pragma once

namespace {

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
  // every lane of column ch now holds the sums; lane (rsub, ch) with rsub <
  // ICOORD writes coordinate ch + rsub*LPR, so the coordinates' epilogues run
  // side by side rather than one after another
  if (rsub < ICOORD) {
    double dqk = dq[0];
#pragma unroll
    for (int k = 1; k < ICOORD; ++k) dqk = rsub == k ? dq[k] : dqk;
    const int i = ch + rsub * G::LPR;
    if (i < 8) {
      if constexpr (!TH) {
        gq[l * 8 + i] = (float)dqk;
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
          const double ir2 = 1.0 / r2, ir3 = ir2 / sqrt(r2);  // 1/r^2, 1/r^3
          const double ds = dls * sc * sc, dqs = dqk * sc * ci;
          ga = ds * a * ir3 - dqs * b * ir2;
          gb = ds * b * ir3 + dqs * a * ir2;
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
// ORD: visit the lookups in the order perm (as k_forward).
// SAVED: the forward's lists (NbrList saved) replace the search.
template <int DT, int M, bool EMIT, bool TH, int KS = NB, bool ORD = false, bool SAVED = false>
__global__ void __launch_bounds__(THREADS) k_backward(const float* __restrict__ q, Params P,
                                                      const void* __restrict__ table,
                                                      const float* __restrict__ gout, float* __restrict__ gtab,
                                                      float* __restrict__ gq, uint32_t* __restrict__ pair_key,
                                                      uint2* __restrict__ pair_val, const uint32_t* __restrict__ gate,
                                                      const uint32_t* __restrict__ perm, NbrList saved) {
  static_assert(!EMIT || KS == NB, "the sorted scatter takes lists of 32");
  static_assert(!(SAVED || ORD) || (KS == NB && !TH), "orders and saved lists serve the k = 32 lookup");
  __shared__ SearchLds<WAVE, KS> S;
  if (gate && merge_chosen(*gate, P.L)) return;
  WaveCtx c;
  if (!wave_ctx(P, c, ORD)) return;
  const int lane = c.lane;
  Search<KS> srch(P, S.tab, S.wave[c.wave], c.wave, lane);
  WaveLds<KS>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  uint32_t my_l = 0;
  if constexpr (ORD)
    my_l = phase_a_perm<TH>(q, perm, c.base, c.nl, P, FR, lane);
  else
    phase_a<TH>(q, c.base, c.nl, P, FR, lane);
  const char* tb = reinterpret_cast<const char*>(table);
  for (int t = 0; t < c.nl; ++t) {
    const Frame& F = FR[t];
    const Sel sel = read_sel(F);
    const int64_t l = ORD ? (int64_t)(uint32_t)__builtin_amdgcn_readlane(my_l, t) : c.base + t;
    int count;
    if constexpr (SAVED)
      count = srch.load(F, sel, 0, saved, l, P.N);
    else
      count = srch.run(F, sel, 0);
    if (!EMIT && gtab && count > 0) scatter_atomic<M, KS>(W, count, gout, l, gtab, lane);
    if (gq && (!ORD || l < P.L)) grad_query<DT, M, TH, KS>(F, W, S.tab, count, tb, gout, l, lane, gq, q, P);
    if (EMIT && gtab && lane < NB && (!ORD || l < P.L)) {
      const int32_t s = W.nbr[0][lane].slot;
      pair_key[l * NB + lane] = s >= 0 ? (uint32_t)s : P.N;
      pair_val[l * NB + lane] = make_uint2((uint32_t)l, __float_as_uint(W.wgt[0][lane]));
    }
    wave_lds_sync();
  }
}

}  // namespace
