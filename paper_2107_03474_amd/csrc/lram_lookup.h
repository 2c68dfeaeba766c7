// lram_lookup.h -- part of liblram (included by lram.hip only).
//
// Lookup kernels: neighbour lists, the forward gather-reduce (pipelined for k
// = 32, chunked for other k).

#pragma once

namespace {

// ---------------------------------------------------------------------------
// Kernels.

struct WaveCtx {
  int wave, lane;
  int64_t base;
  int nl;
};

// xcd: take the workgroups' ranges XCD-contiguously (for lookups visited in a
// locality order, so that neighbouring ranges share an L2).
__device__ __forceinline__ bool wave_ctx(const Params P, WaveCtx& c, bool xcd = false) {
  c.wave = threadIdx.x / WAVE;
  c.lane = threadIdx.x % WAVE;
  const int64_t blk = xcd ? xcd_block() : (int64_t)blockIdx.x;
  c.base = (blk * WAVES + c.wave) * P.lpw;
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
template <int DT, int M, int KS, int R = NB, int NBUF = 1>
__device__ __forceinline__ void fwd_issue(const char* __restrict__ tb, const WaveLds<KS, NBUF>& W, int buf, int lane,
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
template <int DT, int M, int KS, int R = NB, int NBUF = 1>
__device__ __forceinline__ void fwd_accumulate(const WaveLds<KS, NBUF>& W, int buf, int lane,
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

// Sums the row groups of the wave (xor shuffles) and writes out[l] once
// (nothing when !ok: only the store is skipped, so that the row loads are
// waited for on every path and the next lookup's loads need not wait for
// this store).
template <int DT, int M>
__device__ __forceinline__ void fwd_store(int lane, int64_t l, float (&acc)[FwdGeom<DT, M>::EPL],
                                          void* __restrict__ out, bool ok = true) {
  using G = FwdGeom<DT, M>;
  const int rsub = lane / G::LPR, col = lane % G::LPR;
#pragma unroll
  for (int mask = G::LPR; mask < WAVE; mask <<= 1)
#pragma unroll
    for (int e = 0; e < G::EPL; ++e) acc[e] += __shfl_xor(acc[e], mask);
  if (rsub == 0 && ok) {
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
__device__ __forceinline__ void fwd_consume(const WaveLds<NB, 2>& W, int buf, int lane, int64_t l,
                                            const uint32_t (&v)[FwdGeom<DT, M>::NI][FwdGeom<DT, M>::DW],
                                            void* __restrict__ out, bool ok = true) {
  float acc[FwdGeom<DT, M>::EPL];
#pragma unroll
  for (int e = 0; e < FwdGeom<DT, M>::EPL; ++e) acc[e] = 0.0f;
  fwd_accumulate<DT, M, NB>(W, buf, lane, v, acc);
  fwd_store<DT, M>(lane, l, acc, out, ok);
}

// TH: the input is the activation layer's z [L][16] instead of q [L][8]; the
// scale s is folded into the weights by the search.
// ORD: visit the lookups in the order perm (position -> lookup, e.g. sorted
// by closest lattice point, so that lookups sharing rows run close together
// in time and on the same XCD); outputs still go to the lookup's row.
// SAVE: write every lookup's list for the backward (NbrList).
template <int DT, int M, bool TH, bool ORD = false, bool SAVE = false>
__global__ void __launch_bounds__(THREADS) k_forward(const float* __restrict__ q, Params P,
                                                     const void* __restrict__ table, void* __restrict__ out,
                                                     const uint32_t* __restrict__ perm, NbrList save) {
  using G = FwdGeom<DT, M>;
  __shared__ SearchLds<WAVE, NB, 2> S;
  WaveCtx c;
  if (!wave_ctx(P, c, ORD)) return;
  Search<NB, 2> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<NB, 2>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  uint32_t my_l = 0;
  if constexpr (ORD)
    my_l = phase_a_perm<TH>(q, perm, c.base, c.nl, P, FR, c.lane);
  else
    phase_a<TH>(q, c.base, c.nl, P, FR, c.lane);
  const char* tb = reinterpret_cast<const char*>(table);
  uint32_t v[G::NI][G::DW];
  srch.run(FR[0], read_sel(FR[0]), 0);
  fwd_issue<DT, M, NB>(tb, W, 0, c.lane, v);
  for (int t = 0; t < c.nl; ++t) {
    const int buf = t & 1;
    const int64_t l = ORD ? (int64_t)(uint32_t)__builtin_amdgcn_readlane(my_l, t) : c.base + t;
    // search lookup t+1 while the rows of lookup t are in flight
    if (t + 1 < c.nl) srch.run(FR[t + 1], read_sel(FR[t + 1]), buf ^ 1);
    const bool ok = !ORD || l < P.L;
    fwd_consume<DT, M>(W, buf, c.lane, ok ? l : 0, v, out, ok);
    if constexpr (SAVE) srch.save(buf, save, l, ok);
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

}  // namespace
