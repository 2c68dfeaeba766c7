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

template <int DT, int M>
__global__ void __launch_bounds__(THREADS) k_sparse_adam(void* __restrict__ table, int64_t N,
                                                         float* __restrict__ grad, float* __restrict__ m1,
                                                         float* __restrict__ m2, AdamArgs a) {
  constexpr int RW = WAVE / M;  // rows per wave
  const int lane = threadIdx.x % WAVE;
  const int col = lane % M, sub = lane / M;
  // lanes of this lane's row in a wave-wide ballot
  constexpr uint64_t row_mask = M == WAVE ? ~0ull : (1ull << (M % WAVE)) - 1ull;
  const uint64_t seg = row_mask << (M * sub);
  const int64_t waves = (int64_t)gridDim.x * WAVES;
  for (int64_t rb = ((int64_t)blockIdx.x * WAVES + threadIdx.x / WAVE) * RW; rb < N; rb += waves * RW) {
    const int64_t r = rb + sub;
    const bool in = r < N;
    const size_t o = (size_t)(in ? r : 0) * M + col;
    const float g = in ? grad[o] : 0.0f;
    const bool touched = (__ballot(g != 0.0f) & seg) != 0;
    if (in && touched) {
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
}

}  // namespace
