// Head-wise rotation calibration (TurboESM Sec. 3.2): for the post-RoPE keys
// X (ncal x 64) of one head, Pi = V^T where X = U Sigma V^T.
//
// One block per head. The Gram matrix G = X^T X is accumulated in fp64 and
// diagonalized in LDS by cyclic Jacobi rotations in the round-robin
// (tournament) order: each of the 63 rounds of a sweep applies 32 disjoint
// plane rotations at once. Eigenvalues of G are sigma^2; eigenvectors are the
// right singular vectors. Rows of Pi are ordered by descending sigma and
// signed so that each row's largest-magnitude entry is positive (lowest
// index on ties).
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr int kMaxSweeps = 40;
constexpr int kStageRows = 32;

struct CalibSmem {
  double G[kDim * kDim];
  double V[kDim * kDim];
  float xs[kStageRows * kDim];
  double c[kPairs], s[kPairs];
  int p[kPairs], q[kPairs];
  double red[256];
  int rank[kDim];
  int done;
};

__device__ __forceinline__ int tournament_player(int pos, int round) {
  return pos == 0 ? 0 : ((pos - 1 + round) % (kDim - 1)) + 1;
}

__global__ __launch_bounds__(256) void calibrate_kernel(const float* x, int ncal, float* pi_out,
                                                        float* sing_out) {
  __shared__ CalibSmem sm;
  const int head = blockIdx.x;
  const int t = threadIdx.x;
  const float* X = x + (int64_t)head * ncal * kDim;

  // ---- Gram matrix in fp64: thread t owns entries e = t + 256 r
  double acc[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0;
  for (int row0 = 0; row0 < ncal; row0 += kStageRows) {
    const int rows = min(kStageRows, ncal - row0);
    for (int e = t; e < kStageRows * kDim; e += 256)
      sm.xs[e] = (e / kDim < rows) ? X[(int64_t)row0 * kDim + e] : 0.0f;
    __syncthreads();
    for (int rr = 0; rr < rows; ++rr) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int e = t + 256 * r;
        acc[r] = fma((double)sm.xs[rr * kDim + (e >> 6)], (double)sm.xs[rr * kDim + (e & 63)], acc[r]);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int e = t + 256 * r;
    sm.G[e] = acc[r];
    sm.V[e] = ((e >> 6) == (e & 63)) ? 1.0 : 0.0;
  }
  __syncthreads();

  // ---- cyclic Jacobi, round-robin order
  for (int sweep = 0; sweep < kMaxSweeps; ++sweep) {
    // convergence: off-diagonal mass versus diagonal mass
    double off = 0.0, dia = 0.0;
    for (int e = t; e < kDim * kDim; e += 256) {
      const double g = sm.G[e];
      if ((e >> 6) == (e & 63)) dia += g * g; else off += g * g;
    }
    sm.red[t] = off;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (t < w) sm.red[t] += sm.red[t + w];
      __syncthreads();
    }
    const double off_tot = sm.red[0];
    __syncthreads();
    sm.red[t] = dia;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if (t < w) sm.red[t] += sm.red[t + w];
      __syncthreads();
    }
    const double dia_tot = sm.red[0];
    __syncthreads();
    if (off_tot <= 1e-30 * dia_tot || off_tot == 0.0) break;

    for (int round = 0; round < kDim - 1; ++round) {
      if (t < kPairs) {
        int a = tournament_player(t, round), b = tournament_player(kDim - 1 - t, round);
        if (a > b) { const int tmp = a; a = b; b = tmp; }
        const double gpq = sm.G[a * kDim + b];
        double c = 1.0, s = 0.0;
        if (gpq != 0.0) {
          const double tau = (sm.G[b * kDim + b] - sm.G[a * kDim + a]) / (2.0 * gpq);
          double tn;
          if (fabs(tau) > 1e150) {
            tn = 0.5 / tau;
          } else {
            tn = (tau >= 0.0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
          }
          c = 1.0 / sqrt(1.0 + tn * tn);
          s = tn * c;
        }
        sm.p[t] = a; sm.q[t] = b; sm.c[t] = c; sm.s[t] = s;
      }
      __syncthreads();
      // G <- G J (columns p, q)
      for (int e = t; e < kPairs * kDim; e += 256) {
        const int k = e >> 6, r = e & 63;
        const int a = sm.p[k], b = sm.q[k];
        const double c = sm.c[k], s = sm.s[k];
        const double ga = sm.G[r * kDim + a], gb = sm.G[r * kDim + b];
        sm.G[r * kDim + a] = c * ga - s * gb;
        sm.G[r * kDim + b] = s * ga + c * gb;
      }
      __syncthreads();
      // G <- J^T G (rows p, q) and V <- V J (columns p, q)
      for (int e = t; e < kPairs * kDim; e += 256) {
        const int k = e >> 6, r = e & 63;
        const int a = sm.p[k], b = sm.q[k];
        const double c = sm.c[k], s = sm.s[k];
        const double ga = sm.G[a * kDim + r], gb = sm.G[b * kDim + r];
        sm.G[a * kDim + r] = c * ga - s * gb;
        sm.G[b * kDim + r] = s * ga + c * gb;
        const double va = sm.V[r * kDim + a], vb = sm.V[r * kDim + b];
        sm.V[r * kDim + a] = c * va - s * vb;
        sm.V[r * kDim + b] = s * va + c * vb;
      }
      __syncthreads();
    }
  }

  // ---- order by descending eigenvalue, canonical signs, write Pi and sigma
  if (t < kDim) {
    const double lt = sm.G[t * kDim + t];
    int rank = 0;
    for (int b = 0; b < kDim; ++b) {
      const double lb = sm.G[b * kDim + b];
      rank += (lb > lt || (lb == lt && b < t)) ? 1 : 0;
    }
    sm.rank[t] = rank;
    // column t of V is the eigenvector of eigenvalue lt
    int arg = 0;
    double best = -1.0;
    for (int k = 0; k < kDim; ++k) {
      const double v = fabs(sm.V[k * kDim + t]);
      if (v > best) { best = v; arg = k; }
    }
    const double sg = (sm.V[arg * kDim + t] < 0.0) ? -1.0 : 1.0;
    float* dst = pi_out + ((int64_t)head * kDim + rank) * kDim;
    for (int k = 0; k < kDim; ++k) dst[k] = (float)(sg * sm.V[k * kDim + t]);
    if (sing_out) sing_out[(int64_t)head * kDim + rank] = (float)sqrt(lt > 0.0 ? lt : 0.0);
  }
}

hipError_t launch_calibrate(const float* x, int nheads, int ncal, float* pi_out, float* sing_out,
                            hipStream_t st) {
  hipLaunchKernelGGL(calibrate_kernel, dim3(nheads), dim3(256), 0, st, x, ncal, pi_out, sing_out);
  return hipGetLastError();
}

// ------------------------------------------------------- table calibration
// Calibrated 8-level table per head (Sec. 3.3: calibrated, separate K and V
// tables): the 1-D Lloyd iteration (k-means) on every normalized coordinate
// u = 8 x^ / ||x^|| (x^ = Pi x in fp64, x^ = x without Pi; a zero vector
// gives zeros) of the head's calibration vectors. Per iteration: assign each
// u to the level whose midpoint interval holds it (u > t_m strictly counts,
// so a tie goes to the lower level), replace each level by the mean of its
// cell (fp64 sums; an empty cell keeps its level), take the largest level
// change, sort, and stop once that change is below tol, or after max_iter.
//
// One block of 4 waves per head. u is recomputed every iteration (no
// workspace): a wave takes one vector at a time, lane i forming x^_i from
// row i of Pi staged in LDS and the vector staged in LDS, the norm by a wave
// reduction. Every lane owns 8 fp64 bins and counts in LDS; the block sums
// them in a fixed order.
constexpr int kLutWaves = 4;
constexpr int kPiPitch = kDim + 1;       // doubles per staged row of Pi

struct LutSmem {
  double pi[kDim * kPiPitch];
  double xv[kLutWaves][kDim];
  double bsum[kLutWaves * kDim][8];
  int bcnt[kLutWaves * kDim][8];
  double psum[32][8];
  int pcnt[32][8];
  double c[8];
  int done;
};

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void calibrate_lut_kernel(const float* x, int ncal, const float* pi,
                                                            LutInit init, int max_iter, double tol,
                                                            float* lut_out) {
  __shared__ LutSmem sm;
  const int head = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* X = x + (int64_t)head * ncal * kDim;
  const bool rot = pi != nullptr;
  if (rot) {
    const float* P = pi + (int64_t)head * kDim * kDim;
    for (int e = t; e < kDim * kDim; e += 256) sm.pi[(e >> 6) * kPiPitch + (e & 63)] = (double)P[e];
  }
  if (t < 8) sm.c[t] = (double)init.c[t];
  if (t == 0) sm.done = 0;
  __syncthreads();
  double* bs = sm.bsum[wave * kDim + lane];
  int* bc = sm.bcnt[wave * kDim + lane];
  for (int it = 0; it < max_iter; ++it) {
    double th[7];
#pragma unroll
    for (int m = 0; m < 7; ++m) th[m] = 0.5 * (sm.c[m] + sm.c[m + 1]);
#pragma unroll
    for (int m = 0; m < 8; ++m) { bs[m] = 0.0; bc[m] = 0; }
    for (int v = wave; v < ncal; v += kLutWaves) {
      const double xi = (double)X[(int64_t)v * kDim + lane];
      double xh = xi;
      if (rot) {
        sm.xv[wave][lane] = xi;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const double* row = sm.pi + lane * kPiPitch;
        xh = 0.0;
#pragma unroll 8
        for (int k = 0; k < kDim; ++k) xh = fma(row[k], sm.xv[wave][k], xh);
      }
      const double n2 = wave_sum_f64(xh * xh);
      const double u = (n2 > 0.0) ? xh * (8.0 / sqrt(n2)) : 0.0;
      int m = 0;
#pragma unroll
      for (int k = 0; k < 7; ++k) m += (u > th[k]) ? 1 : 0;
      bs[m] += u;
      bc[m] += 1;
      if (rot) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // xv is rewritten next
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
    }
    __syncthreads();
    {
      // 32 partials per level: thread (part, m) sums 8 lanes' bins in order
      const int m = t & 7, part = t >> 3;
      double sacc = 0.0;
      int cacc = 0;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        sacc += sm.bsum[part * 8 + r][m];
        cacc += sm.bcnt[part * 8 + r][m];
      }
      sm.psum[part][m] = sacc;
      sm.pcnt[part][m] = cacc;
    }
    __syncthreads();
    if (t == 0) {
      double cn[8], delta = 0.0;
      for (int m = 0; m < 8; ++m) {
        double sacc = 0.0;
        int cacc = 0;
        for (int part = 0; part < 32; ++part) { sacc += sm.psum[part][m]; cacc += sm.pcnt[part][m]; }
        cn[m] = (cacc > 0) ? sacc / (double)cacc : sm.c[m];
        delta = fmax(delta, fabs(cn[m] - sm.c[m]));
      }
      for (int i = 1; i < 8; ++i) {          // insertion sort, ascending
        const double key = cn[i];
        int j = i - 1;
        while (j >= 0 && cn[j] > key) { cn[j + 1] = cn[j]; --j; }
        cn[j + 1] = key;
      }
      for (int m = 0; m < 8; ++m) sm.c[m] = cn[m];
      sm.done = (delta < tol) ? 1 : 0;
    }
    __syncthreads();
    if (sm.done) break;
  }
  if (t < 8) lut_out[(int64_t)head * 8 + t] = (float)sm.c[t];
}

hipError_t launch_calibrate_lut(const float* x, int nheads, int ncal, const float* pi, const float* init,
                                int max_iter, double tol, float* lut_out, hipStream_t st) {
  LutInit in;
  for (int m = 0; m < 8; ++m) in.c[m] = init[m];
  hipLaunchKernelGGL(calibrate_lut_kernel, dim3(nheads), dim3(256), 0, st, x, ncal, pi, in, max_iter, tol,
                     lut_out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- ebar
// Per-head mean absolute residual of the per-element correction (Sec. 3.4,
// Eq. 7): over every normalized coordinate u = 8 x^ / ||x^|| of the head's
// calibration vectors (computed as in calibrate_lut_kernel), the mean of
// |u - c[idx]| with idx = #{m : u > (c_m + c_{m+1})/2} (fp64 midpoints of the
// fp32 levels). Each lane sums its coordinates in fp64 in vector order; the
// 256 lane sums are added in a fixed order. A head whose table is not
// strictly ascending gets NaN.
struct EbarSmem {
  double pi[kDim * kPiPitch];
  double xv[kLutWaves][kDim];
  double red[256];
};

__global__ __launch_bounds__(256) void calibrate_ebar_kernel(const float* x, int ncal, const float* pi,
                                                             const float* lut, float* ebar_out, int stride) {
  __shared__ EbarSmem sm;
  const int head = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* X = x + (int64_t)head * ncal * kDim;
  const bool rot = pi != nullptr;
  if (rot) {
    const float* P = pi + (int64_t)head * kDim * kDim;
    for (int e = t; e < kDim * kDim; e += 256) sm.pi[(e >> 6) * kPiPitch + (e & 63)] = (double)P[e];
  }
  double c[8];
#pragma unroll
  for (int m = 0; m < 8; ++m) c[m] = (double)lut[(int64_t)head * 8 + m];
  bool asc = true;
#pragma unroll
  for (int m = 0; m < 7; ++m) asc = asc && (c[m] < c[m + 1]);
  double th[7];
#pragma unroll
  for (int m = 0; m < 7; ++m) th[m] = 0.5 * (c[m] + c[m + 1]);
  __syncthreads();
  double acc = 0.0;
  for (int v = wave; v < ncal; v += kLutWaves) {
    const double xi = (double)X[(int64_t)v * kDim + lane];
    double xh = xi;
    if (rot) {
      sm.xv[wave][lane] = xi;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const double* row = sm.pi + lane * kPiPitch;
      xh = 0.0;
#pragma unroll 8
      for (int k = 0; k < kDim; ++k) xh = fma(row[k], sm.xv[wave][k], xh);
    }
    const double n2 = wave_sum_f64(xh * xh);
    const double u = (n2 > 0.0) ? xh * (8.0 / sqrt(n2)) : 0.0;
    double lv = c[0];
#pragma unroll
    for (int k = 0; k < 7; ++k) lv = (u > th[k]) ? c[k + 1] : lv;
    acc += fabs(u - lv);
    if (rot) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");   // xv is rewritten next
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
  sm.red[t] = acc;
  __syncthreads();
  if (t == 0) {
    double total = 0.0;
    for (int i = 0; i < 256; ++i) total += sm.red[i];
    const double mean = total / ((double)ncal * kDim);
    ebar_out[(int64_t)head * stride] = asc ? (float)mean : __int_as_float(0x7FC00000);
  }
}

hipError_t launch_calibrate_ebar(const float* x, int nheads, int ncal, const float* pi, const float* lut,
                                 float* ebar_out, int stride, hipStream_t st) {
  hipLaunchKernelGGL(calibrate_ebar_kernel, dim3(nheads), dim3(256), 0, st, x, ncal, pi, lut, ebar_out,
                     stride);
  return hipGetLastError();
}

}  // namespace tq
