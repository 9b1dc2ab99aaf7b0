// Audio-Visual Budget Allocation (AVBA, Sec. 3.2 of the OmniMem paper).
//
//  avba_partials  per (layer, KV head): fp64 sums over visual and audio
//                 rows of a, a ln a and s (the inputs of Eqs. 9, 10, 13).
//  avba_allocate  one workgroup: normalised entropies and mean cosines,
//                 compressibilities C_v, C_a, C^(l), the split w_v (Eq. 11),
//                 layer shares B_tot softmax(C^(l)/T) (Eq. 14) clamped to
//                 [B_min, B_max] with the sum kept (water-filling on the
//                 scale kappa), largest-remainder integer budgets and the
//                 per-modality split.  All in fp64.
//                 Offline budgets (end of Sec. 3.2: fixed in advance from a
//                 calibration set) use the same kernel in three more modes:
//                 adding a step's C^(l) to the calibration sums, turning
//                 their means into layer budgets by the same Eq. (14) path
//                 (no token count caps them), and a step under given layer
//                 budgets, which only caps them at N_l and splits them.
#include "common.h"

namespace omnimem {

namespace {

constexpr int kStatSets = 2;  // visual, audio (the layer set is their union)


constexpr int kPartThreads = 256;
constexpr int kPartRows = 512;   // rows per partial-sum workgroup

__host__ __device__ inline int part_chunks(const Dims& dm) {
  return (int)((dm.max_tokens + kPartRows - 1) / kPartRows);
}

// stat_part[l][g][chunk][set][0..3] = {sum a, sum a ln a, sum s, count}
// over the visual (set 0) and audio (set 1) rows of one chunk of layer l,
// KV head g.
__global__ __launch_bounds__(kPartThreads) void avba_partials(const LayerDesc* __restrict__ layers, Dims dm,
                                                              const float* __restrict__ a,
                                                              const float* __restrict__ s,
                                                              double* __restrict__ part) {
  const int l = blockIdx.z, g = blockIdx.y, chunk = blockIdx.x;
  const int N = layers[l].n;
  const uint8_t* mod = layers[l].mod;
  const float* ag = a + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const float* sg = s + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  double acc[kStatSets * 4] = {};
  const int j1 = min(N, (chunk + 1) * kPartRows);
  // the thread's rows (j, j + 256, ...), all requested before the first sum
  constexpr int kPer = kPartRows / kPartThreads;
  static_assert(kPer * kPartThreads == kPartRows, "whole rows per thread");
  float xa[kPer], xs[kPer];
  int xm[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int j = chunk * kPartRows + u * kPartThreads + (int)threadIdx.x;
    xa[u] = j < j1 ? ag[j] : 0.0f;
    xs[u] = j < j1 ? sg[j] : 0.0f;
    xm[u] = j < j1 ? (int)mod[j] : -1;
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    if (xm[u] < 0) continue;
    const int o = xm[u] ? 4 : 0;
    const double x = xa[u];
    acc[o + 0] += x;
    acc[o + 1] += x > 0.0 ? x * log(x) : 0.0;
    acc[o + 2] += xs[u];
    acc[o + 3] += 1.0;
  }
  // all eight sums reduced together: wave shuffles, then one LDS round
  __shared__ double wsum[kPartThreads / 64][kStatSets * 4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < kStatSets * 4; ++q) {
    double v = acc[q];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) wsum[wave][q] = v;
  }
  __syncthreads();
  if (threadIdx.x < kStatSets * 4) {
    double t = 0.0;
    for (int w = 0; w < kPartThreads / 64; ++w) t += wsum[w][threadIdx.x];
    part[(((int64_t)l * dm.Hkv + g) * part_chunks(dm) + chunk) * kStatSets * 4 + threadIdx.x] = t;
  }
}

// Normalised entropy of x / sum x over K entries from sum x and sum x ln x:
// H = ln S - (sum x ln x) / S, divided by ln K; 0 when K <= 1 or S == 0.
__device__ inline double norm_entropy(double sum, double xlogx, double count) {
  if (count <= 1.0 || sum <= 0.0) return 0.0;
  return (log(sum) - xlogx / sum) / log(count);
}

constexpr int kMaxLayers = 1024;
constexpr int kMaxSums = 2048;   // L * H_kv * 8 partial sums kept in LDS
constexpr int kAllocThreads = 1024;  // the per-head entropies take fp64 logs: all the lanes of a CU

enum AllocMode : int {
  kOnline = 0,       // Eq. (14) from this step's statistics, then the split
  kCalibAdd = 1,     // calib[l] (+)= this step's C^(l); nothing else written
  kFixed = 2,        // layer budgets given: capped at N_l, then the split
  kCalibFinish = 3,  // layer budgets from calib[l] / steps (no statistics read)
};

// calib: [L] calibration sums; calib_first: a kCalibAdd step that starts
// them (assigns instead of adding); steps: their count (kCalibFinish).
// layer_budgets: read in kFixed, written in kCalibFinish.
__global__ __launch_bounds__(kAllocThreads) void avba_allocate(const LayerDesc* __restrict__ layers, Dims dm,
                                                     const double* __restrict__ part, int64_t total,
                                                     float ratio_r, float temperature, float bmin_frac,
                                                     float bmax_frac, int mode, double* __restrict__ calib,
                                                     int calib_first, double steps,
                                                     int32_t* __restrict__ layer_budgets,
                                                     int32_t* __restrict__ budgets, float* __restrict__ stats) {
  __shared__ double c_l[kMaxLayers], w_v[kMaxLayers], p[kMaxLayers], x[kMaxLayers];
  __shared__ int n_l[kMaxLayers], k_v[kMaxLayers], lo[kMaxLayers], hi[kMaxLayers], b_l[kMaxLayers];
  __shared__ double s_kappa;
  __shared__ double bk[2 * kMaxLayers], bf[2 * kMaxLayers];  // breakpoints and f there
  __shared__ double sums[kMaxSums];
  __shared__ double ent[kMaxSums / (kStatSets * 4) * 3];  // per (layer, head): visual, audio, layer
  const int L = dm.L;
  const double B = (double)total;
  const double T = (double)temperature;
  const double r = (double)ratio_r;

  if (mode == kCalibFinish) {
    // the mean compressibility of each layer; counts that never bind
    for (int l = threadIdx.x; l < L; l += blockDim.x) {
      c_l[l] = calib[l] / steps;
      n_l[l] = 0x7fffffff;
      k_v[l] = 0;
      w_v[l] = 0.0;
    }
    __syncthreads();
  } else {
  // --- chunk partials summed per (layer, head, quantity), in chunk order;
  // sixteen chunks' loads in flight at a time ---
  const int nchunk = part_chunks(dm);
  for (int x = threadIdx.x; x < L * dm.Hkv * kStatSets * 4; x += blockDim.x) {
    const int lg = x / (kStatSets * 4), q = x % (kStatSets * 4);
    const double* src = part + (int64_t)lg * nchunk * kStatSets * 4 + q;
    double t = 0.0;
    for (int c0 = 0; c0 < nchunk; c0 += 16) {
      double v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = c0 + u < nchunk ? src[(c0 + u) * kStatSets * 4] : 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u) t += v[u];
    }
    sums[x] = t;
  }
  __syncthreads();

  // --- per-layer statistics (Eqs. 9, 10, 13); the normalised entropies of
  // every (layer, head, set) first, in parallel ---
  for (int q = threadIdx.x; q < L * dm.Hkv * 3; q += blockDim.x) {
    const double* P = sums + (q / 3) * kStatSets * 4;
    const int set = q % 3;
    ent[q] = set == 0 ? norm_entropy(P[0], P[1], P[3])
                      : set == 1 ? norm_entropy(P[4], P[5], P[7])
                                 : norm_entropy(P[0] + P[4], P[1] + P[5], P[3] + P[7]);
  }
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += blockDim.x) {
    double hv = 0.0, ha = 0.0, hl = 0.0, sv = 0.0, sa = 0.0, cnt_v = 0.0, cnt_a = 0.0;
    for (int g = 0; g < dm.Hkv; ++g) {
      const double* P = sums + (l * dm.Hkv + g) * kStatSets * 4;
      const double* E = ent + (l * dm.Hkv + g) * 3;
      hv += E[0];
      ha += E[1];
      hl += E[2];
      sv += P[2];
      sa += P[6];
      cnt_v = P[3];
      cnt_a = P[7];
    }
    hv /= dm.Hkv; ha /= dm.Hkv; hl /= dm.Hkv;
    const double sbar_v = cnt_v > 0.0 ? sv / (dm.Hkv * cnt_v) : 0.0;
    const double sbar_a = cnt_a > 0.0 ? sa / (dm.Hkv * cnt_a) : 0.0;
    const double sbar_l = (cnt_v + cnt_a) > 0.0 ? (sv + sa) / (dm.Hkv * (cnt_v + cnt_a)) : 0.0;
    const double cv = hv * (1.0 - sbar_v), ca = ha * (1.0 - sbar_a), cl = hl * (1.0 - sbar_l);
    const double den = cv * r + ca;
    const double wv = den > 0.0 ? cv * r / den : r / (r + 1.0);
    c_l[l] = cl;
    w_v[l] = wv;
    n_l[l] = layers[l].n;
    k_v[l] = (int)cnt_v;
    if (stats) {
      float* o = stats + (int64_t)l * 10;
      o[0] = (float)hv; o[1] = (float)ha; o[2] = (float)hl;
      o[3] = (float)sbar_v; o[4] = (float)sbar_a; o[5] = (float)sbar_l;
      o[6] = (float)cv; o[7] = (float)ca; o[8] = (float)cl; o[9] = (float)wv;
    }
  }
  __syncthreads();
  }  // statistics of this step

  if (mode == kCalibAdd) {
    for (int l = threadIdx.x; l < L; l += blockDim.x) calib[l] = calib_first ? c_l[l] : calib[l] + c_l[l];
    return;
  }
  if (mode == kFixed) {
    for (int l = threadIdx.x; l < L; l += blockDim.x) b_l[l] = min(max(layer_budgets[l], 0), n_l[l]);
    __syncthreads();
  } else {

  // --- Eq. (14): softmax over layers of C / T (exps in parallel, the max
  // and the sum in layer order), bounds ---
  if (threadIdx.x == 0) {
    double mx = -INFINITY;
    for (int l = 0; l < L; ++l) mx = fmax(mx, c_l[l] / T);
    s_kappa = mx;
  }
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += blockDim.x) p[l] = exp(c_l[l] / T - s_kappa);
  __syncthreads();
  if (threadIdx.x == 0) {
    double sum = 0.0;
    for (int l = 0; l < L; ++l) sum += p[l];
    s_kappa = sum;
  }
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += blockDim.x) p[l] /= s_kappa;
  const int lo_base = (int)ceil(((double)bmin_frac * B) / L);
  const int hi_base = (int)floor(((double)bmax_frac * B) / L);
  for (int l = threadIdx.x; l < L; l += blockDim.x) {
    lo[l] = min(lo_base, n_l[l]);
    hi[l] = min(hi_base, n_l[l]);
  }
  __syncthreads();
  double sum_hi = 0.0;
  for (int l = 0; l < L; ++l) sum_hi += hi[l];

  if (sum_hi <= B) {
    for (int l = threadIdx.x; l < L; l += blockDim.x) { x[l] = hi[l]; b_l[l] = hi[l]; }
    __syncthreads();
  } else {
    // --- water-fill: kappa with sum_l clamp(kappa B p_l, lo_l, hi_l) = B ---
    // Breakpoints kappa = lo_l / (B p_l) and hi_l / (B p_l); f is
    // non-decreasing and linear in between.  Each thread evaluates f at its
    // breakpoints (summing over layers in order); kappa interpolates between
    // the first breakpoint where f reaches B and the breakpoint before it.
    auto f = [&](double kap) {
      double t = 0.0;
      for (int l = 0; l < L; ++l) t += fmin(fmax(kap * B * p[l], (double)lo[l]), (double)hi[l]);
      return t;
    };
    for (int q = threadIdx.x; q < 2 * L; q += blockDim.x) {
      const int l = q >> 1;
      const double kb = p[l] > 0.0 ? ((q & 1) ? hi[l] : lo[l]) / (B * p[l]) : INFINITY;
      bk[q] = kb;
      bf[q] = kb < INFINITY ? f(kb) : INFINITY;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double k_hi = INFINITY, f_hi = 0.0;
      for (int q = 0; q < 2 * L; ++q)
        if (bf[q] >= B && bk[q] < k_hi) { k_hi = bk[q]; f_hi = bf[q]; }
      double k_lo = -INFINITY, f_lo = 0.0;
      for (int q = 0; q < 2 * L; ++q)
        if (bk[q] < k_hi && bk[q] > k_lo) { k_lo = bk[q]; f_lo = bf[q]; }
      double kap = 0.0;
      if (k_hi < INFINITY) kap = k_lo > -INFINITY ? k_lo + (B - f_lo) * (k_hi - k_lo) / (f_hi - f_lo) : k_hi;
      s_kappa = kap;
    }
    __syncthreads();
    const double kap = s_kappa;
    for (int l = threadIdx.x; l < L; l += blockDim.x) {
      x[l] = fmin(fmax(kap * B * p[l], (double)lo[l]), (double)hi[l]);
      b_l[l] = (int)floor(x[l]);
    }
    __syncthreads();
    // --- largest remainder: leftover units to the largest fractional parts
    // among layers below their upper bound, ties to the lower layer ---
    double fl_sum = 0.0;
    for (int l = 0; l < L; ++l) fl_sum += b_l[l];
    const int leftover = (int)(B - fl_sum);
    __syncthreads();
    for (int l = threadIdx.x; l < L; l += blockDim.x) {
      if (b_l[l] >= hi[l]) continue;
      const double fr = x[l] - floor(x[l]);
      int rank = 0;
      for (int m = 0; m < L; ++m) {
        if (m == l || floor(x[m]) >= hi[m]) continue;
        const double fm = x[m] - floor(x[m]);
        if (fm > fr || (fm == fr && m < l)) ++rank;
      }
      if (rank < leftover) b_l[l] += 1;
    }
    __syncthreads();
  }
  }  // layer budgets of Eq. (14)
  if (mode == kCalibFinish) {
    for (int l = threadIdx.x; l < L; l += blockDim.x) layer_budgets[l] = b_l[l];
    return;
  }

  // --- per-modality split (Eqs. 11-12) ---
  for (int l = threadIdx.x; l < L; l += blockDim.x) {
    const int bl = b_l[l];
    const int kv = k_v[l], ka = n_l[l] - k_v[l];
    int mv = (int)floor(w_v[l] * bl + 0.5);
    mv = min(max(mv, max(0, bl - ka)), min(kv, bl));
    budgets[2 * l] = mv;
    budgets[2 * l + 1] = bl - mv;
  }
}

// Partial sums over a and s for the allocation kernel.
void launch_sums(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a, const float* s,
                 hipStream_t st) {
  OMNIMEM_LAUNCH(ws, K_AVBA_PART, st,
                 avba_partials<<<dim3(part_chunks(dm), dm.Hkv, dm.L), kPartThreads, 0, st>>>(desc, dm, a, s,
                                                                                            ws.stat_part));
}

}  // namespace

int allocate_part_chunks(const Dims& dm) { return part_chunks(dm); }

hipError_t launch_allocate(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a,
                           const float* s, int64_t total, float ratio_r, float temperature, float bmin_frac,
                           float bmax_frac, int32_t* budgets, float* stats, hipStream_t st) {
  launch_sums(dm, desc, ws, a, s, st);
  OMNIMEM_LAUNCH(ws, K_AVBA_ALLOC, st,
                 avba_allocate<<<1, kAllocThreads, 0, st>>>(desc, dm, ws.stat_part, total, ratio_r, temperature,
                                                            bmin_frac, bmax_frac, kOnline, nullptr, 0, 0.0, nullptr,
                                                            budgets, stats));
  return hipGetLastError();
}

hipError_t launch_calibrate(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a,
                            const float* s, float ratio_r, bool first, float* stats, hipStream_t st) {
  launch_sums(dm, desc, ws, a, s, st);
  OMNIMEM_LAUNCH(ws, K_AVBA_ALLOC, st,
                 avba_allocate<<<1, kAllocThreads, 0, st>>>(desc, dm, ws.stat_part, 0, ratio_r, 1.0f, 0.0f,
                                                            0.0f, kCalibAdd, ws.calib, first ? 1 : 0, 0.0, nullptr,
                                                            nullptr, stats));
  return hipGetLastError();
}

hipError_t launch_calibration_budgets(const Dims& dm, const Workspace& ws, int64_t total, float temperature,
                                      float bmin_frac, float bmax_frac, int steps, int32_t* layer_budgets,
                                      hipStream_t st) {
  OMNIMEM_LAUNCH(ws, K_AVBA_ALLOC, st,
                 avba_allocate<<<1, kAllocThreads, 0, st>>>(nullptr, dm, nullptr, total, 1.0f,
                                                            temperature, bmin_frac, bmax_frac, kCalibFinish, ws.calib,
                                                            0, (double)steps, layer_budgets, nullptr, nullptr));
  return hipGetLastError();
}

hipError_t launch_allocate_fixed(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const float* a,
                                 const float* s, const int32_t* layer_budgets, float ratio_r, int32_t* budgets,
                                 float* stats, hipStream_t st) {
  launch_sums(dm, desc, ws, a, s, st);
  OMNIMEM_LAUNCH(ws, K_AVBA_ALLOC, st,
                 avba_allocate<<<1, kAllocThreads, 0, st>>>(desc, dm, ws.stat_part, 0, ratio_r, 1.0f, 0.0f,
                                                            0.0f, kFixed, nullptr, 0, 0.0,
                                                            const_cast<int32_t*>(layer_budgets), budgets, stats));
  return hipGetLastError();
}

}  // namespace omnimem
