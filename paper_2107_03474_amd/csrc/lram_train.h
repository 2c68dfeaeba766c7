// lram_train.h -- part of liblram (included by lram.hip only).
//
// Training-side companions: access statistics and the Adam step on touched
// rows.

#pragma once

namespace {

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

// touched[s] = 1 for every location s in a lookup's list of its closest 32
// (the rows a backward of these lookups writes): plain byte stores, every
// writer stores the same value.
__global__ void __launch_bounds__(THREADS) k_mark_touched(const float* __restrict__ q, Params P,
                                                          uint8_t* __restrict__ touched) {
  __shared__ SearchLds<WAVE> S;
  WaveCtx c;
  if (!wave_ctx(P, c)) return;
  Search<NB> srch(P, S.tab, S.wave[c.wave], c.wave, c.lane);
  WaveLds<NB>& W = S.wave[c.wave];
  Frame* FR = S.frames[c.wave];
  phase_a<false>(q, c.base, c.nl, P, FR, c.lane);
  for (int t = 0; t < c.nl; ++t) {
    const int count = srch.run(FR[t], read_sel(FR[t]), 0);
    if (c.lane < count) touched[W.nbr[0][c.lane].slot] = 1;
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

// One row's Adam update (M lanes, lane = column) when its gradient row is not
// identically zero; the gradient row is then cleared.  seg: this lane's row's
// lanes in a wave-wide ballot (every lane of the wave takes part).
template <int DT, int M>
__device__ __forceinline__ void adam_row(void* __restrict__ table, float* __restrict__ grad, float* __restrict__ m1,
                                         float* __restrict__ m2, const AdamArgs& a, int64_t r, bool in, int col,
                                         uint64_t seg) {
  const size_t o = (size_t)(in ? r : 0) * M + col;
  const float g = in ? grad[o] : 0.0f;
  const bool nonzero = (__ballot(g != 0.0f) & seg) != 0;
  if (in && nonzero) {
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

template <int M>
constexpr uint64_t row_lanes() { return M == WAVE ? ~0ull : (1ull << (M % WAVE)) - 1ull; }

template <int DT, int M>
__global__ void __launch_bounds__(THREADS) k_sparse_adam(void* __restrict__ table, int64_t N,
                                                         float* __restrict__ grad, float* __restrict__ m1,
                                                         float* __restrict__ m2, AdamArgs a) {
  constexpr int RW = WAVE / M;  // rows per wave
  const int lane = threadIdx.x % WAVE;
  const int col = lane % M, sub = lane / M;
  const uint64_t seg = row_lanes<M>() << (M * sub);
  const int64_t waves = (int64_t)gridDim.x * WAVES;
  for (int64_t rb = ((int64_t)blockIdx.x * WAVES + threadIdx.x / WAVE) * RW; rb < N; rb += waves * RW) {
    const int64_t r = rb + sub;
    adam_row<DT, M>(table, grad, m1, m2, a, r, r < N, col, seg);
  }
}

// The same step on the rows whose flag in touched [N] is set (by
// k_mark_touched for the step's lookups): a wave reads 64 flags at once and
// updates only the flagged rows (RW at a time), so the step reads N bytes of
// flags plus the flagged rows instead of the whole N x M gradient; flags are
// cleared.  A flagged row whose gradient is identically zero keeps value and
// moments, as in k_sparse_adam.
template <int DT, int M>
__global__ void __launch_bounds__(THREADS) k_sparse_adam_touched(void* __restrict__ table, int64_t N,
                                                                 float* __restrict__ grad, float* __restrict__ m1,
                                                                 float* __restrict__ m2, uint8_t* __restrict__ touched,
                                                                 AdamArgs a) {
  constexpr int RW = WAVE / M;
  const int lane = threadIdx.x % WAVE;
  const int col = lane % M, sub = lane / M;
  const uint64_t seg = row_lanes<M>() << (M * sub);
  const int64_t waves = (int64_t)gridDim.x * WAVES;
  for (int64_t base = ((int64_t)blockIdx.x * WAVES + threadIdx.x / WAVE) * WAVE; base < N; base += waves * WAVE) {
    const bool flag = base + lane < N && touched[base + lane] != 0;
    uint64_t mask = __ballot(flag);
    if (flag) touched[base + lane] = 0;
    while (mask) {
      // the wave's next RW flagged rows, one per group of M lanes
      int pick = -1;
#pragma unroll
      for (int k = 0; k < RW; ++k) {
        const int b = mask ? (int)__builtin_ctzll(mask) : -1;
        mask &= mask - 1;
        pick = k == sub ? b : pick;
      }
      adam_row<DT, M>(table, grad, m1, m2, a, base + pick, pick >= 0, col, seg);
    }
  }
}

}  // namespace
