// Select and compact (Eqs. 4, 5 and 8 of the OmniMem paper).
//
//  psi_topk        one workgroup per (layer, KV head, modality): psi =
//                  a^lambda (1 - s) as an order-preserving 32-bit key,
//                  radix select of the M-th largest key (4 passes of 8 bits,
//                  LDS histogram), then an ordered ballot/prefix-sum pass
//                  that keeps every key above the threshold and the first
//                  ones equal to it (ties to the lower row), emitting rows
//                  in ascending order.
//  gather_compact  k_out[g][i] = k[g][idx[g][i]] and the same for v, 16 bytes
//                  per lane, whole 256-byte rows per 16 lanes.
#include "common.h"

namespace omnimem {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kLdsKeys = 32768;   // member keys of a segment held in LDS (128 KB)
constexpr int kBins = 2048;       // radix digit of up to 11 bits

__device__ inline uint32_t psi_key(float a, float s, float lambda) {
  s = fminf(1.0f, fmaxf(-1.0f, s));
  const float w = lambda == 0.0f ? 1.0f : (a > 0.0f ? powf(a, lambda) : 0.0f);
  float psi = w * (1.0f - s);
  if (!(psi >= 0.0f)) psi = 0.0f;  // NaN or negative inputs rank last
  return __float_as_uint(psi + 0.0f);  // +0 for -0: nonnegative floats order as uints
}

// Exclusive prefix of `flag` over the block in thread order; *total gets the
// block's count.  Uses wave_tot[kSelWaves] and two barriers.
__device__ inline int block_prefix(bool flag, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long bal = __ballot(flag);
  const int before = __popcll(bal & ((1ull << lane) - 1ull));
  __syncthreads();
  if (lane == 0) wave_tot[wave] = __popcll(bal);
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int c = wave_tot[w];
    base += w < wave ? c : 0;
    tot += c;
  }
  *total = tot;
  return base + before;
}

// Inclusive prefix sum of v over the 64 lanes.
__device__ inline int wave_inclusive(int v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

__global__ __launch_bounds__(kSelThreads) void psi_topk(const LayerDesc* __restrict__ layers, Dims dm, float lambda,
                                                        const float* __restrict__ a, const float* __restrict__ s,
                                                        const int32_t* __restrict__ budgets,
                                                        uint32_t* __restrict__ keys, int32_t* __restrict__ idx,
                                                        int* __restrict__ eff) {
  __shared__ uint32_t skey[kLdsKeys];
  __shared__ int hist[kBins];
  __shared__ int wave_tot[kSelWaves];
  __shared__ int s_bin, s_need;

  const int mu = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
  const int N = layers[l].n;
  const uint8_t* mod = layers[l].mod;
  const int64_t off = ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const float* ag = a + off;
  const float* sg = s + off;
  uint32_t* kg = keys + off;   // keys by working-set row
  int32_t* ig = idx + off;

  // Pass 0: keys of this modality's rows, by row in global memory and by
  // member rank in LDS.
  int K = 0;
  for (int t0 = 0; t0 < N; t0 += kSelThreads) {
    const int j = t0 + threadIdx.x;
    const bool member = j < N && (mod[j] ? 1 : 0) == mu;
    int cnt;
    const int rank = K + block_prefix(member, wave_tot, &cnt);
    if (member) {
      const uint32_t key = psi_key(ag[j], sg[j], lambda);
      kg[j] = key;
      if (rank < kLdsKeys) skey[rank] = key;
    }
    K += cnt;
  }
  const int M = min(max(budgets[2 * l + mu], 0), K);
  const int Kv = mu ? N - K : K;
  const int Mv = mu ? min(max(budgets[2 * l], 0), Kv) : M;
  if (g == 0 && threadIdx.x == 0) eff[2 * l + mu] = M;
  const int out0 = mu ? Mv : 0;
  const bool in_lds = K <= kLdsKeys;
  __syncthreads();

  // Radix select of the M-th largest key, digits of 11, 11 and 10 bits.
  uint32_t thr = 0;
  int take_eq = 0;
  const bool all = M >= K;
  if (!all && M > 0) {
    uint32_t prefix = 0, mask = 0;
    int need = M;
    for (int pass = 0; pass < 3; ++pass) {
      const int shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
      const uint32_t dmask = pass == 2 ? 1023u : 2047u;
      for (int b = threadIdx.x; b < kBins; b += kSelThreads) hist[b] = 0;
      __syncthreads();
      if (in_lds) {
        for (int r = threadIdx.x; r < K; r += kSelThreads) {
          const uint32_t key = skey[r];
          if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1);
        }
      } else {
        for (int j = threadIdx.x; j < N; j += kSelThreads) {
          if ((mod[j] ? 1 : 0) != mu) continue;
          const uint32_t key = kg[j];
          if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1);
        }
      }
      __syncthreads();
      // Counts above each bin, from the top: thread t owns bins 2047-2t, 2046-2t.
      const int b1 = kBins - 1 - 2 * (int)threadIdx.x, b2 = b1 - 1;
      const int h1 = hist[b1], h2 = hist[b2];
      const int incl = wave_inclusive(h1 + h2);
      const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
      if (lane == 63) wave_tot[wave] = incl;
      __syncthreads();
      int above = incl - (h1 + h2);
      for (int w = 0; w < wave; ++w) above += wave_tot[w];
      if (above < need && need <= above + h1) { s_bin = b1; s_need = need - above; }
      else if (above + h1 < need && need <= above + h1 + h2) { s_bin = b2; s_need = need - above - h1; }
      __syncthreads();
      prefix |= (uint32_t)s_bin << shift;
      mask |= dmask << shift;
      need = s_need;
      __syncthreads();
    }
    thr = prefix;
    take_eq = need;
  }

  // Ordered emission: rows above the threshold and the first `take_eq` rows
  // equal to it, in ascending row order.
  int eq_seen = 0, emitted = 0;
  for (int t0 = 0; t0 < N; t0 += kSelThreads) {
    const int j = t0 + threadIdx.x;
    const bool member = j < N && (mod[j] ? 1 : 0) == mu;
    const uint32_t key = member ? kg[j] : 0u;
    const bool eq = member && !all && key == thr;
    int eq_tot;
    const int eq_rank = eq_seen + block_prefix(eq, wave_tot, &eq_tot);
    const bool sel = member && (all || (M > 0 && (key > thr || (eq && eq_rank < take_eq))));
    int sel_tot;
    const int rank = emitted + block_prefix(sel, wave_tot, &sel_tot);
    if (sel) ig[out0 + rank] = j;
    eq_seen += eq_tot;
    emitted += sel_tot;
  }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void gather_compact(const LayerDesc* __restrict__ layers, Dims dm,
                                                      const int32_t* __restrict__ idx, const int* __restrict__ eff) {
  constexpr int CPR = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  constexpr int RPP = 256 / CPR;                // rows per pass
  constexpr int ROWS = 64;                      // rows per workgroup
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int M = eff[2 * l] + eff[2 * l + 1];
  const int i0 = blockIdx.x * ROWS;
  if (i0 >= M) return;
  const int32_t* ig = idx + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const T* v = reinterpret_cast<const T*>(Ld.v) + (int64_t)g * Ld.kv_hs;
  T* ko = reinterpret_cast<T*>(Ld.k_out) + (int64_t)g * Ld.out_hs;
  T* vo = reinterpret_cast<T*>(Ld.v_out) + (int64_t)g * Ld.out_hs;
  const int sub = threadIdx.x % CPR;
  for (int r = threadIdx.x / CPR; r < ROWS; r += RPP) {
    const int i = i0 + r;
    if (i >= M) break;
    const int src = ig[i];
    if ((unsigned)src >= (unsigned)Ld.n) continue;  // never read outside the working set
    const uint4 kx = *reinterpret_cast<const uint4*>(k + (int64_t)src * Ld.kv_rs + sub * (16 / sizeof(T)));
    const uint4 vx = *reinterpret_cast<const uint4*>(v + (int64_t)src * Ld.kv_rs + sub * (16 / sizeof(T)));
    *reinterpret_cast<uint4*>(ko + (int64_t)i * Ld.out_rs + sub * (16 / sizeof(T))) = kx;
    *reinterpret_cast<uint4*>(vo + (int64_t)i * Ld.out_rs + sub * (16 / sizeof(T))) = vx;
  }
}

template <typename T, int D>
void launch_gather(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const int32_t* idx, hipStream_t st) {
  dim3 grid((unsigned)((dm.max_tokens + 63) / 64), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_GATHER, st, gather_compact<T, D><<<grid, 256, 0, st>>>(desc, dm, idx, ws.eff));
}

}  // namespace

hipError_t launch_select_compact(const Dims& dm, int dtype, float lambda, const LayerDesc* desc,
                                 const Workspace& ws, const float* a, const float* s, const int32_t* budgets,
                                 int32_t* idx, hipStream_t st) {
  int32_t* ix = idx ? idx : ws.idx;
  OMNIMEM_LAUNCH(ws, K_TOPK, st, psi_topk<<<dim3(2, dm.Hkv, dm.L), kSelThreads, 0, st>>>(desc, dm, lambda, a, s, budgets, ws.keys, ix, ws.eff));
  if (dtype == 0) {
    if (dm.d == 128) launch_gather<uint16_t, 128>(dm, desc, ws, ix, st);
    else launch_gather<uint16_t, 64>(dm, desc, ws, ix, st);
  } else {
    if (dm.d == 128) launch_gather<float, 128>(dm, desc, ws, ix, st);
    else launch_gather<float, 64>(dm, desc, ws, ix, st);
  }
  return hipGetLastError();
}

}  // namespace omnimem
