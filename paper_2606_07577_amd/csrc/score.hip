// Accumulated attention importance a_k (Eq. 6 of the OmniMem paper).
//
// a[g][j] sums, over every chunk query i of every query head h of KV head
// g, the softmax probability A[h][i][j] of the chunk attention (Eq. 1:
// one softmax over both caches and the visible chunk rows).  A row of A is
// only known once its normaliser is, so the work is two passes over the
// score matrix S = scale * Q K^T, both on MFMA tiles:
//   lse_pass     per (head, query, key range): running max and sum of
//                exp2 over the range (ranges split long rows over more
//                workgroups so that small layers still fill the chip)
//   colsum_pass  merges the range partials into the normaliser of each
//                query, then per (head, key): sum_i exp(S[i][j] - lse[i])
//   head_sum     a[g][j] = sum over the G query heads of KV head g.
// Scores stay in registers; nothing of size queries x keys touches HBM.
// Both passes stream one operand through double-buffered LDS (next tile
// prefetched into registers while the current one is consumed) and keep
// the other in registers, 64 rows per wavefront.  lse_merge joins them.
#include "common.h"

namespace omnimem {

namespace {

constexpr int kThreads = 256;       // 4 wavefronts
constexpr int kRowsPerWave = 64;    // register-resident rows per wave (two 32-wide MFMA blocks)
constexpr int kBlockRows = 4 * kRowsPerWave;
constexpr int kTile = 64;           // streamed rows per LDS stage

__device__ inline float wave_xor32(float x) { return __shfl_xor(x, 32, 64); }

__device__ inline float max16(const floatx16& v) {
  float a = fmaxf(fmaxf(v[0], v[1]), v[2]);
  float b = fmaxf(fmaxf(v[3], v[4]), v[5]);
  float c = fmaxf(fmaxf(v[6], v[7]), v[8]);
  float d = fmaxf(fmaxf(v[9], v[10]), v[11]);
  float e = fmaxf(fmaxf(v[12], v[13]), v[14]);
  return fmaxf(fmaxf(fmaxf(a, b), fmaxf(c, d)), fmaxf(e, v[15]));
}

// Register prefetch of one LDS stage: kTile rows of D elements.
template <typename T, int D>
struct Stage {
  static constexpr int CPR = D * (int)sizeof(T) / 16;           // 16-byte chunks per row
  static constexpr int PER_THREAD = kTile * CPR / kThreads;     // chunks per thread
  static constexpr int LD = D + lds_pad<T>();
  uint4 r[PER_THREAD];

  // Rows at or past `valid` (>= 1) repeat the last valid row: the loads
  // need no branch and no wait, and consumers mask those rows out.
  __device__ inline void load(const T* src, int64_t row_stride, int valid) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = threadIdx.x + i * kThreads;
      const int row = c / CPR, x = c % CPR;
      r[i] = gload16(src + (int64_t)min(row, valid - 1) * row_stride + x * (16 / sizeof(T)));
    }
  }
  __device__ inline void store(T* lds) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int c = threadIdx.x + i * kThreads;
      const int row = c / CPR, x = c % CPR;
      *reinterpret_cast<uint4*>(lds + row * LD + x * (16 / sizeof(T))) = r[i];
    }
  }
};

// Pass 1: for the 256 queries [q0, q0+256) of head h and the keys
// [kr0, kr1) of one range, the per-query running max m and sum l of
// exp2(scale_log2 * q.k), merged over both lanes that share a query.
// MFMA tile: rows = 32 keys (A from LDS), columns = 32 queries (B in
// registers); each lane owns one query and 16 of its keys per tile.
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void lse_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                        float2* __restrict__ part) {
  using M = Mfma<T>;
  using S = Stage<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = S::LD;
  __shared__ __attribute__((aligned(16))) T ktile[2][kTile * LD];

  const int l = blockIdx.z / dm.Hq, h = blockIdx.z % dm.Hq;
  const LayerDesc Ld = layers[l];
  if (Ld.lse_in) return;
  const int C = Ld.n_chunk, N = Ld.n, nc = Ld.n_cache;
  const int q0 = blockIdx.y * kBlockRows;
  if (q0 >= C) return;
  const int kend_blk = dm.causal ? min(N, nc + min(q0 + kBlockRows, C)) : N;
  const int kr0 = blockIdx.x * dm.krange;
  if (kr0 >= kend_blk) return;
  const int kr1 = min(kr0 + dm.krange, kend_blk);

  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const int qw = q0 + wave * kRowsPerWave;
  const bool active = qw < C;
  const int kend_wave = min(kr1, dm.causal ? min(N, nc + min(qw + kRowsPerWave, C)) : N);

  typename M::frag qf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int my_q = qw + cb * 32 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      qf[cb][ks] = my_q < C ? M::gload(q + (int64_t)my_q * Ld.q_rs + ks * M::KSTEP + half * M::PER_LANE)
                            : M::zero();
  }
  const float sl2 = Ld.scale_log2;
  float m[2] = {-1e30f, -1e30f}, lsum[2] = {0.0f, 0.0f};

  S pre;
  pre.load(k + (int64_t)kr0 * Ld.kv_rs, Ld.kv_rs, min(kTile, N - kr0));
  pre.store(ktile[0]);
  __syncthreads();
  int buf = 0;
  for (int t = kr0; t < kr1; t += kTile, buf ^= 1) {
    const bool has_next = t + kTile < kr1;
    if (has_next) pre.load(k + (int64_t)(t + kTile) * Ld.kv_rs, Ld.kv_rs, min(kTile, N - t - kTile));
    if (active && t < kend_wave) {
      floatx16 acc[2][2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = floatx16{};
      const T* a0 = ktile[buf] + (lane & 31) * LD + half * M::PER_LANE;
      const T* a1 = a0 + 32 * LD;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const typename M::frag f0 = M::load(a0 + ks * M::KSTEP);
        const typename M::frag f1 = M::load(a1 + ks * M::KSTEP);
        acc[0][0] = M::mma(f0, qf[0][ks], acc[0][0]);
        acc[0][1] = M::mma(f0, qf[1][ks], acc[0][1]);
        acc[1][0] = M::mma(f1, qf[0][ks], acc[1][0]);
        acc[1][1] = M::mma(f1, qf[1][ks], acc[1][1]);
      }
#pragma unroll
      for (int cb = 0; cb < 2; ++cb) {
        const int qcb = qw + cb * 32;
        // masking only where the tile passes the range or some query's horizon;
        // key t + off (off = rb*32 + acc_row(r, lane) - half*4, a constant) is
        // visible iff off <= lim
        if (t + kTile > kend_wave || (dm.causal && t + kTile - 1 - nc > qcb)) {
          const int base = t + half * 4;
          int lim = kend_wave - 1 - base;
          if (dm.causal) lim = min(lim, qcb + (lane & 31) + nc - base);
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int off = rb * 32 + (r >> 2) * 8 + (r & 3);
              acc[rb][cb][r] = off <= lim ? acc[rb][cb][r] : -INFINITY;
            }
        }
        const float mx = fmaxf(max16(acc[0][cb]), max16(acc[1][cb])) * sl2;
        const float mnew = fmaxf(m[cb], mx);
        const float neg = -mnew;
        float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s0 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[0][cb][r], sl2, neg));
          s1 += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[1][cb][r], sl2, neg));
        }
        lsum[cb] = lsum[cb] * __builtin_amdgcn_exp2f(m[cb] - mnew) + (s0 + s1);
        m[cb] = mnew;
      }
    }
    if (has_next) pre.store(ktile[buf ^ 1]);
    __syncthreads();
  }
  if (!active) return;
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const float m2 = wave_xor32(m[cb]), l2 = wave_xor32(lsum[cb]);
    const float mt = fmaxf(m[cb], m2);
    const float lt = lsum[cb] * __builtin_amdgcn_exp2f(m[cb] - mt) + l2 * __builtin_amdgcn_exp2f(m2 - mt);
    const int my_q = qw + cb * 32 + (lane & 31);
    if (half == 0 && my_q < C)
      part[(((int64_t)l * dm.Hq + h) * dm.n_kr + blockIdx.x) * dm.max_chunk + my_q] = make_float2(mt, lt);
  }
}

// Normaliser of every chunk query in log2 units: the caller's lse, or the
// merge of the key-range partials covering the query's visible keys.
// Also writes the natural-log value to lse_out when requested.
__global__ __launch_bounds__(256) void lse_merge(const LayerDesc* __restrict__ layers, Dims dm,
                                                 const float2* __restrict__ part, float* __restrict__ lse2,
                                                 float* __restrict__ lse_out) {
  const int l = blockIdx.z, h = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= Ld.n_chunk) return;
  const int64_t o = ((int64_t)l * dm.Hq + h) * dm.max_chunk + i;
  if (Ld.lse_in) {
    const float v = Ld.lse_in[(int64_t)h * Ld.n_chunk + i];
    lse2[o] = v * kLog2e;
    if (lse_out) lse_out[o] = v;
    return;
  }
  const float2* p = part + ((int64_t)l * dm.Hq + h) * dm.n_kr * dm.max_chunk + i;
  const int vis = dm.causal ? min(Ld.n, Ld.n_cache + i + 1) : Ld.n;
  const int nr = (vis + dm.krange - 1) / dm.krange;
  // one pass, online: (mx, sum) of the ranges seen so far
  float mx = -1e30f, sum = 0.0f;
#pragma unroll 4
  for (int r = 0; r < nr; ++r) {
    const float2 v = p[(int64_t)r * dm.max_chunk];
    const float m2 = fmaxf(mx, v.x);
    sum = sum * __builtin_amdgcn_exp2f(mx - m2) + v.y * __builtin_amdgcn_exp2f(v.x - m2);
    mx = m2;
  }
  const float v2 = mx + __log2f(sum);
  lse2[o] = v2;
  if (lse_out) lse_out[o] = v2 * kLn2;
}

// Pass 2: per-query-head column sums colsum[h][j] = sum_i exp(S[i][j] -
// lse[i]) for the 256 keys [k0, k0+256).  MFMA tile: rows = 32 queries (A
// from LDS), columns = 32 keys (B in registers, two blocks per wave); each
// lane accumulates one key's sum over 16 query rows per tile. 
template <typename T, int D>
__global__ __launch_bounds__(kThreads, 2) void colsum_pass(const LayerDesc* __restrict__ layers, Dims dm,
                                                           const float* __restrict__ lse2_all,
                                                           float* __restrict__ colsum) {
  using M = Mfma<T>;
  using S = Stage<T, D>;
  constexpr int NKS = D / M::KSTEP;
  constexpr int LD = S::LD;
  __shared__ __attribute__((aligned(16))) T qtile[2][kTile * LD];
  __shared__ __attribute__((aligned(16))) float lse2[2][kTile];

  const int l = blockIdx.z, h = blockIdx.y / dm.n_qc, qc = blockIdx.y % dm.n_qc;
  const LayerDesc Ld = layers[l];
  const int N = Ld.n, nc = Ld.n_cache;
  const int k0 = blockIdx.x * kBlockRows;
  if (k0 >= N) return;
  // this workgroup's slice of the chunk queries
  const int C = min(Ld.n_chunk, (qc + 1) * dm.qchunk);
  const int qlo = qc * dm.qchunk;
  const int wave = wave_id(), lane = threadIdx.x & 63, half = lane >> 5;
  const int g = h / dm.G;
  const T* q = reinterpret_cast<const T*>(Ld.q) + (int64_t)h * Ld.q_hs;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const float* lse2_lh = lse2_all + ((int64_t)l * dm.Hq + h) * dm.max_chunk;
  const int kw = k0 + wave * kRowsPerWave;
  const bool active = kw < N;

  typename M::frag kf[2][NKS];
#pragma unroll
  for (int cb = 0; cb < 2; ++cb) {
    const int key = kw + cb * 32 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      kf[cb][ks] = key < N ? M::gload(k + (int64_t)key * Ld.kv_rs + ks * M::KSTEP + half * M::PER_LANE)
                           : M::zero();
  }
  // First query seeing any key of the block (chunk row nc + t is seen by i >= t).
  const int qstart = max(qlo, dm.causal ? (max(0, k0 - nc) / kTile) * kTile : 0);
  const int qfirst_wave = dm.causal ? max(0, kw - nc) : 0;
  const float sl2 = Ld.scale_log2;
  float cs[2] = {0.0f, 0.0f};

  // normaliser of tile row threadIdx.x (+inf past the chunk: probability 0)
  auto load_lse = [&](int qt) {
    const int i = qt + (int)threadIdx.x;
    return (threadIdx.x < kTile && i < C) ? gload<float>(lse2_lh + i) : INFINITY;
  };

  S pre;
  float pre_lse = INFINITY;
  if (qstart < C) {
    pre.load(q + (int64_t)qstart * Ld.q_rs, Ld.q_rs, min(kTile, C - qstart));
    pre.store(qtile[0]);
    if (threadIdx.x < kTile) lse2[0][threadIdx.x] = load_lse(qstart);
  }
  __syncthreads();
  int buf = 0;
  for (int qt = qstart; qt < C; qt += kTile, buf ^= 1) {
    const bool has_next = qt + kTile < C;
    if (has_next) {
      pre.load(q + (int64_t)(qt + kTile) * Ld.q_rs, Ld.q_rs, min(kTile, C - qt - kTile));
      pre_lse = load_lse(qt + kTile);
    }
    if (active && qt + kTile > qfirst_wave) {
      floatx16 acc[2][2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) acc[rb][cb] = floatx16{};
      const T* a0 = qtile[buf] + (lane & 31) * LD + half * M::PER_LANE;
      const T* a1 = a0 + 32 * LD;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const typename M::frag f0 = M::load(a0 + ks * M::KSTEP);
        const typename M::frag f1 = M::load(a1 + ks * M::KSTEP);
        acc[0][0] = M::mma(f0, kf[0][ks], acc[0][0]);
        acc[0][1] = M::mma(f0, kf[1][ks], acc[0][1]);
        acc[1][0] = M::mma(f1, kf[0][ks], acc[1][0]);
        acc[1][1] = M::mma(f1, kf[1][ks], acc[1][1]);
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        // lse2 of the 16 query rows this lane holds: 4 runs of 4 rows
        float nl[16];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const floatx4 v = *reinterpret_cast<const floatx4*>(&lse2[buf][rb * 32 + j * 8 + half * 4]);
          nl[j * 4 + 0] = -v[0]; nl[j * 4 + 1] = -v[1]; nl[j * 4 + 2] = -v[2]; nl[j * 4 + 3] = -v[3];
        }
        const int qb = qt + rb * 32;
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
          float sum = 0.0f;
          if (dm.causal && kw + cb * 32 + 31 - nc > qb) {
            // chunk key t = key - nc is seen by query qb + acc_row(r) iff
            // (r >> 2) * 8 + (r & 3) >= t - qb - half * 4
            const int dlim = kw + cb * 32 + (lane & 31) - nc - qb - half * 4;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][cb][r], sl2, nl[r]));
              sum += ((r >> 2) * 8 + (r & 3)) >= dlim ? p : 0.0f;
            }
          } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) sum += __builtin_amdgcn_exp2f(__builtin_fmaf(acc[rb][cb][r], sl2, nl[r]));
          }
          cs[cb] += sum;
        }
      }
    }
    if (has_next) {
      pre.store(qtile[buf ^ 1]);
      if (threadIdx.x < kTile) lse2[buf ^ 1][threadIdx.x] = pre_lse;
    }
    __syncthreads();
  }
  if (!active) return;
  cs[0] += wave_xor32(cs[0]);
  cs[1] += wave_xor32(cs[1]);
  float* out = colsum + (((int64_t)l * dm.Hq + h) * dm.n_qc + qc) * dm.max_tokens;
  const int key = kw + half * 32 + (lane & 31);
  if (key < N) out[key] = half ? cs[1] : cs[0];
}

// a[l][g][j] = sum over the G query heads of KV head g and the query
// slices, in a fixed order.
__global__ void head_sum(const LayerDesc* __restrict__ layers, Dims dm, const float* __restrict__ colsum,
                         float* __restrict__ a) {
  const int l = blockIdx.z, g = blockIdx.y;
  const int N = layers[l].n;
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= N) return;
  const float* p = colsum + ((int64_t)l * dm.Hq + (int64_t)g * dm.G) * dm.n_qc * dm.max_tokens + j;
  const int n = dm.G * dm.n_qc;
  float sum = 0.0f;
  int x = 0;
  for (; x + 8 <= n; x += 8) {  // eight independent loads in flight
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = p[(int64_t)(x + u) * dm.max_tokens];
#pragma unroll
    for (int u = 0; u < 8; ++u) sum += v[u];
  }
  for (; x < n; ++x) sum += p[(int64_t)x * dm.max_tokens];
  a[((int64_t)l * dm.Hkv + g) * dm.max_tokens + j] = sum;
}

template <typename T, int D>
void launch_typed(const Dims& dm, const LayerDesc* desc, const Workspace& ws, float* lse_out, float* a,
                  hipStream_t st) {
  const unsigned qblocks = (unsigned)((dm.max_chunk + kBlockRows - 1) / kBlockRows);
  dim3 g1((unsigned)dm.n_kr, qblocks, (unsigned)(dm.L * dm.Hq));
  OMNIMEM_LAUNCH(ws, K_LSE, st, lse_pass<T, D><<<g1, kThreads, 0, st>>>(desc, dm, ws.lse_part));
  dim3 g2((unsigned)((dm.max_tokens + kBlockRows - 1) / kBlockRows), (unsigned)(dm.Hq * dm.n_qc), dm.L);
  dim3 gm((unsigned)((dm.max_chunk + 255) / 256), dm.Hq, dm.L);
  OMNIMEM_LAUNCH(ws, K_LSE_MERGE, st, lse_merge<<<gm, 256, 0, st>>>(desc, dm, ws.lse_part, ws.lse2, lse_out));
  OMNIMEM_LAUNCH(ws, K_COLSUM, st, colsum_pass<T, D><<<g2, kThreads, 0, st>>>(desc, dm, ws.lse2, ws.part));
  dim3 g3((unsigned)((dm.max_tokens + 255) / 256), dm.Hkv, dm.L);
  OMNIMEM_LAUNCH(ws, K_HEADSUM, st, head_sum<<<g3, 256, 0, st>>>(desc, dm, ws.part, a));
}

}  // namespace

// Work split of both passes: key ranges of the LSE pass and query slices of
// the column-sum pass, each only as fine as needed to give the chip about
// 3072 workgroups (ranges never below 512 keys, slices never below 256
// queries; both multiples of the 64-row stage).
void choose_key_ranges(Dims* dm) {
  const int64_t want = 3072;
  auto split = [&](int64_t base, int64_t len, int64_t min_len, int* out_len, int* out_n) {
    const int64_t most = std::max<int64_t>(1, len / min_len);
    const int64_t n = std::min(std::max<int64_t>(1, (want + base - 1) / base), most);
    int64_t piece = (len + n - 1) / n;
    piece = (piece + kTile - 1) / kTile * kTile;
    *out_len = (int)piece;
    *out_n = (int)((len + piece - 1) / piece);
  };
  const int64_t qblocks = (dm->max_chunk + kBlockRows - 1) / kBlockRows;
  split(qblocks * dm->Hq * dm->L, dm->max_tokens, 512, &dm->krange, &dm->n_kr);
  const int64_t kblocks = (dm->max_tokens + kBlockRows - 1) / kBlockRows;
  split(kblocks * dm->Hq * dm->L, dm->max_chunk, 256, &dm->qchunk, &dm->n_qc);
}

hipError_t launch_score(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws,
                        float* lse_out, float* a, int /*unused*/, hipStream_t st) {
  if (dtype == 0) {
    if (dm.d == 128) launch_typed<uint16_t, 128>(dm, desc, ws, lse_out, a, st);
    else launch_typed<uint16_t, 64>(dm, desc, ws, lse_out, a, st);
  } else {
    if (dm.d == 128) launch_typed<float, 128>(dm, desc, ws, lse_out, a, st);
    else launch_typed<float, 64>(dm, desc, ws, lse_out, a, st);
  }
  return hipGetLastError();
}

}  // namespace omnimem
