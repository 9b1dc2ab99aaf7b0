// Select and compact (Eqs. 4, 5 and 8 of the OmniMem paper).
//
//  psi_topk        one workgroup per (layer, KV head, modality): psi =
//                  a^lambda (1 - s) as an order-preserving 32-bit key per
//                  member row (rows dealt to waves in contiguous spans, read
//                  coalesced), radix select of the M-th largest key (12-bit
//                  digits below the bits all keys share, LDS histogram;
//                  the last few candidates ranked directly against each
//                  other), then an ordered emission that keeps every key above the
//                  threshold and the first ones equal to it (ties to the
//                  lower row), in ascending row order, placed by ballots and
//                  block-wide scans.
//  topk_hist, topk_bin, topk_emit
//                  the same selection split over several workgroups per
//                  (layer, KV head) for long working sets (described
//                  where they are defined).
//  gather_compact  k_out[g][i] = k[g][idx[g][i]] and the same for v, 16 bytes
//                  per lane, whole rows per lane group.
#include "../../include/omnimem.h"
#include "common.h"

namespace omnimem {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kLdsKeys = 32768;   // member keys of a segment held in LDS (128 KB)
constexpr int kDigit = 12;        // radix digit bits
constexpr int kBins = 1 << kDigit;
constexpr int kListMax = 256;     // threshold-bin keys ranked directly instead of by more passes

// a^lambda as exp2(lambda * log2 a) on the hardware transcendentals (about
// 1e-7 relative error, far inside the ordering tolerance of the selection).
__device__ inline uint32_t psi_key(float a, float s, float lambda) {
  s = fminf(1.0f, fmaxf(-1.0f, s));
  const float w = lambda == 0.0f ? 1.0f : (a > 0.0f ? __builtin_amdgcn_exp2f(lambda * __builtin_amdgcn_logf(a)) : 0.0f);
  float psi = w * (1.0f - s);
  if (!(psi >= 0.0f)) psi = 0.0f;  // NaN or negative inputs rank last
  return __float_as_uint(psi + 0.0f);  // +0 for -0: nonnegative floats order as uints
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

// Exclusive prefix of the per-wave values v (taken from lane 0) over the
// block in wave order; *total gets the sum.  One barrier; each call site
// passes its own wave_tot array, so no barrier is needed before the writes.
__device__ inline int wave_scan(int v, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_tot[wave] = v;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int c = wave_tot[w];
    base += w < wave ? c : 0;
    tot += c;
  }
  *total = tot;
  return base;
}

// Inclusive scans over the workgroup's threads in thread order (one
// barrier); wsum holds kSelWaves ints per value and must not be reused before a later
// barrier.  tot: the sums.
template <int NV>
__device__ inline void block_inclusive(int (&v)[NV], int (*wsum)[kSelWaves], int (&tot)[NV]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    v[i] = wave_inclusive(v[i]);
    if (lane == 63) wsum[i][wave] = v[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    int base = 0, t = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const int c = wsum[i][w];
      base += w < wave ? c : 0;
      t += c;
    }
    v[i] += base;
    tot[i] = t;
  }
}

// Of PER bins h[0..PER) taken from the highest down, with `above` keys in
// the bins before them and above < need <= above + sum(h): the bin i that
// holds the need-th largest key, how many of its keys are needed and its
// count.  Branch-free: a selection per bin.
template <int PER>
__device__ inline void crossing_bin(const int (&h)[PER], int above, int need, int& bin, int& need_in, int& cnt) {
  bin = 0;
  need_in = 0;
  cnt = 0;
  bool found = false;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const bool hit = !found && need <= above + h[i];
    bin = hit ? i : bin;
    need_in = hit ? need - above : need_in;
    cnt = hit ? h[i] : cnt;
    found = found || hit;
    above += h[i];
  }
}

// Rows are dealt to waves in contiguous spans: wave w owns rows
// [w * 64R, (w + 1) * 64R), and step i of the wave covers the 64 consecutive
// rows w * 64R + 64 i + lane, so every load is coalesced.  Member ranks come
// from ballots within the wave and one scan of the wave totals; the members'
// keys sit at their ranks in LDS (or, for segments too large for LDS, by row
// in global memory).
// SHARED: one workgroup per (layer, modality) ranks rows by the layer's
// importance and redundancy (a and s as reduced over the KV heads by
// layer_inputs, [L][max_tokens] each) and writes the kept rows to every
// head's idx row.
template <bool SHARED>
__global__ __launch_bounds__(kSelThreads) void psi_topk(const LayerDesc* __restrict__ layers, Dims dm, float lambda,
                                                        const float* __restrict__ a, const float* __restrict__ s,
                                                        const int32_t* __restrict__ budgets,
                                                        uint32_t* __restrict__ keys, int32_t* __restrict__ idx,
                                                        int* __restrict__ eff, int* __restrict__ slot_of,
                                                        int* __restrict__ ctl) {
  __shared__ uint32_t skey[kLdsKeys];
  __shared__ int hist[kBins];
  __shared__ int wave_tot[kSelWaves];
  __shared__ int s_bin, s_need, s_cnt, s_lcnt;
  __shared__ uint32_t s_thr;
  __shared__ int wt_mem[kSelWaves], wt_eq[kSelWaves], wt_sel[kSelWaves];
  __shared__ uint32_t wmin[kSelWaves], wmax[kSelWaves];

  const int mu = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
  const int N = layers[l].n;
  const uint8_t* mod = layers[l].mod;
  const int cap = layers[l].out_cap;           // rows per head of the output
  const bool want_slots = layers[l].inplace != 0 && slot_of != nullptr;
  if (ctl != nullptr && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0)
    ctl[1] = 0;  // staging rows needed beyond the reserve, this call
  const int64_t off = ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const float* ag = a + (SHARED ? (int64_t)l * dm.max_tokens : off);
  const float* sg = s + (SHARED ? (int64_t)l * dm.max_tokens : off);
  uint32_t* kg = keys + off;   // keys by working-set row (segments past LDS)
  int32_t* ig = idx + off;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int R = (N + kSelThreads - 1) / kSelThreads;   // rows per lane
  const int wrow0 = wave * 64 * R;
  auto member = [&](int j) { return j < N && (mod[j] ? 1 : 0) == mu; };
  auto read_a = [&](int j) { return gload<float>(ag + j); };
  auto read_s = [&](int j) { return gload<float>(sg + j); };
  // the segment's budget (and the visual one, where the audio rows go),
  // requested first so that their latency overlaps the reads below
  const int bud_mu = budgets[2 * l + mu], bud_v = budgets[2 * l];

  // Membership of this lane's rows (bit i: row wrow0 + 64 i + lane), read in
  // groups of 8 steps so their loads are in flight together; with more than
  // 64 rows per lane the flags are re-read where needed.  With at most one
  // group (R <= 8) the rows' a and s are read in the same round and the
  // keys kept in registers.
  constexpr int kGrp = 8;
  const bool bits_ok = R <= 64;
  const bool one_grp = R <= kGrp;
  unsigned long long mbits = 0;
  int wcount = 0;
  uint32_t kreg[kGrp];
  for (int i0 = 0; i0 < R; i0 += kGrp) {
    // branch-free reads (index clamped into the working set), all issued
    // before the first use
    int mv[kGrp];
    float av[kGrp], sv[kGrp];
    bool mb[kGrp];
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int j = min(wrow0 + (i0 + u) * 64 + lane, N - 1);
      mv[u] = gload<uint8_t>(mod + j);
      if (one_grp) {
        av[u] = read_a(j);
        sv[u] = read_s(j);
      }
    }
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      pin(mv[u]);
      mb[u] = i0 + u < R && wrow0 + (i0 + u) * 64 + lane < N && (mv[u] ? 1 : 0) == mu;
    }
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      wcount += __popcll(__ballot(mb[u]));
      if (mb[u] && i0 + u < 64) mbits |= 1ull << (i0 + u);
      if (one_grp) kreg[u] = psi_key(av[u], sv[u], lambda);
    }
  }
  auto member_at = [&](int i, int j) { return bits_ok ? ((mbits >> i) & 1ull) != 0 : member(j); };
  int K;
  const int rank_base = wave_scan(wcount, wt_mem, &K);
  const bool in_lds = K <= kLdsKeys;
  // keys at their ranks, and the range they span
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  for (int i0 = 0, run = rank_base; i0 < R; i0 += kGrp) {
    bool mb[kGrp];
    float av[kGrp], sv[kGrp];
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int j = wrow0 + (i0 + u) * 64 + lane;
      mb[u] = i0 + u < R && member_at(i0 + u, j);
      if (!one_grp) {
        av[u] = read_a(min(j, N - 1));
        sv[u] = read_s(min(j, N - 1));
      }
    }
    if (!one_grp) {
#pragma unroll
      for (int u = 0; u < kGrp; ++u) { pin(av[u]); pin(sv[u]); }
    }
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const unsigned long long bal = __ballot(mb[u]);
      if (mb[u]) {
        const uint32_t key = one_grp ? kreg[u] : psi_key(av[u], sv[u], lambda);
        kmin = min(kmin, key);
        kmax = max(kmax, key);
        if (in_lds) skey[run + __popcll(bal & lt)] = key;
        else kg[wrow0 + (i0 + u) * 64 + lane] = key;
      }
      run += __popcll(bal);
    }
  }
  // Budgets as applied: each modality's within its rows, visual first
  // within the output capacity, audio in what remains.
  const int Kv = mu ? N - K : K;
  const int Mv = min(min(max(bud_v, 0), Kv), cap);
  const int M = mu ? min(min(max(bud_mu, 0), K), cap - Mv) : Mv;
  if (g == 0 && threadIdx.x == 0) eff[2 * l + mu] = M;
  const int out0 = mu ? Mv : 0;

  // Bits shared by every key (keys of psi in a narrow range share sign,
  // exponent and leading mantissa bits): the radix digits start below them,
  // which spreads the first histogram over its bins instead of piling its
  // atomics onto a few.
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
  }
  if (lane == 0) { wmin[wave] = kmin; wmax[wave] = kmax; }
  __syncthreads();  // keys and their range
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) { kmin = min(kmin, wmin[w]); kmax = max(kmax, wmax[w]); }
  const int width = (kmin ^ kmax) ? 32 - __clz(kmin ^ kmax) : 0;  // low bits in which keys differ

  // Radix select of the M-th largest key over those bits, kDigit at a time.
  uint32_t thr = 0;
  int take_eq = 0, n_eq = K;  // keys equal to the threshold (all of them when none differ)
  const bool all = M >= K;
  if (!all && M > 0) {
    uint32_t prefix = kmin & ~((width < 32 ? (1u << width) : 0u) - 1u), mask = ~((width < 32 ? (1u << width) : 0u) - 1u);
    int need = M;
    for (int top = width; top > 0; top -= kDigit) {
      const int shift = max(0, top - kDigit);
      const uint32_t dmask = (1u << (top - shift)) - 1u;
      for (int b = threadIdx.x; b < kBins; b += kSelThreads) hist[b] = 0;
      if (threadIdx.x == 0) s_lcnt = 0;
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
      // Counts above each bin, from the top: thread t owns the kPer bins
      // below kBins - 1 - kPer t.
      constexpr int kPer = kBins / kSelThreads;
      const int btop = kBins - 1 - kPer * (int)threadIdx.x;
      int h[kPer], mine_h = 0;
#pragma unroll
      for (int u = 0; u < kPer; ++u) { h[u] = hist[btop - u]; mine_h += h[u]; }
      const int incl = wave_inclusive(mine_h);
      if (lane == 63) wave_tot[wave] = incl;
      __syncthreads();
      int above = incl - mine_h;
      for (int w = 0; w < wave; ++w) above += wave_tot[w];
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        if (above < need && need <= above + h[u]) { s_bin = btop - u; s_need = need - above; s_cnt = h[u]; }
        above += h[u];
      }
      __syncthreads();
      prefix |= (uint32_t)s_bin << shift;
      mask |= dmask << shift;
      need = s_need;
      n_eq = s_cnt;
      __syncthreads();
      if (shift > 0 && in_lds && n_eq <= kListMax) {
        // Few keys left in the threshold's bin: collect them (the histogram's
        // memory is free now) and rank each against the others, instead of
        // further passes over all keys.  The key with need - 1 candidates
        // strictly above it, counting its equals, is the threshold.
        int* cand = hist;
        for (int r0 = 0; r0 < K; r0 += kSelThreads) {
          const int r = r0 + (int)threadIdx.x;
          const uint32_t key = r < K ? skey[r] : 0u;
          const bool m = r < K && (key & mask) == prefix;
          const unsigned long long b = __ballot(m);
          int base = 0;
          if (lane == 0 && b) base = atomicAdd(&s_lcnt, __popcll(b));
          base = __shfl(base, 0, 64);
          if (m) cand[base + __popcll(b & lt)] = (int)key;
        }
        __syncthreads();
        if ((int)threadIdx.x < n_eq) {
          const uint32_t c = (uint32_t)cand[threadIdx.x];
          int gt = 0, eq = 0;
          for (int u = 0; u < n_eq; ++u) {
            const uint32_t x = (uint32_t)cand[u];
            gt += x > c ? 1 : 0;
            eq += x == c ? 1 : 0;
          }
          // every candidate equal to the threshold writes the same values
          if (gt < need && need <= gt + eq) { s_thr = c; s_need = need - gt; s_cnt = eq; }
        }
        __syncthreads();
        prefix = s_thr;
        need = s_need;
        n_eq = s_cnt;
        break;
      }
    }
    thr = prefix;
    take_eq = need;
  }

  // Ordered emission: rows above the threshold and the first `take_eq` rows
  // equal to it (ties to the lower row), in ascending row order.  Ranks
  // among the equal keys are needed only when some of them are dropped.
  const bool pick = !all && M > 0;
  const bool eq_ranks = pick && n_eq > take_eq;
  // Keys of steps i0 .. i0+kGrp-1 (members only), read together.
  auto group_keys = [&](int i0, int run, uint32_t (&kk)[kGrp], unsigned long long (&bal)[kGrp]) {
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int j = wrow0 + (i0 + u) * 64 + lane;
      const bool mb = i0 + u < R && member_at(i0 + u, j);
      bal[u] = __ballot(mb);
      kk[u] = mb ? (one_grp ? kreg[u] : (in_lds ? skey[run + __popcll(bal[u] & lt)] : kg[j])) : 0u;
      run += __popcll(bal[u]);
    }
    return run;
  };
  int eq_base = 0;
  if (eq_ranks) {  // uniform: every wave takes this branch or none
    int weq = 0;
    for (int i0 = 0, run = rank_base; i0 < R; i0 += kGrp) {
      uint32_t kk[kGrp];
      unsigned long long bal[kGrp];
      run = group_keys(i0, run, kk, bal);
#pragma unroll
      for (int u = 0; u < kGrp; ++u) weq += __popcll(__ballot(((bal[u] >> lane) & 1ull) && kk[u] == thr));
    }
    int eq_tot;
    eq_base = wave_scan(weq, wt_eq, &eq_tot);
  }
  // selection bits of this lane's rows (bit i; past 64 steps they are
  // recomputed in the writing pass)
  unsigned long long sbits = 0;
  int wsel = 0;
  auto select_group = [&](int i0, int run, int& eqr, unsigned long long (&sb)[kGrp]) {
    uint32_t kk[kGrp];
    unsigned long long bal[kGrp];
    run = group_keys(i0, run, kk, bal);
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const bool mb = (bal[u] >> lane) & 1ull;
      const bool eq = pick && mb && kk[u] == thr;
      const unsigned long long eqb = eq_ranks ? __ballot(eq) : 0ull;
      const bool sel = mb && (all || (pick && (kk[u] > thr || (eq && (!eq_ranks || eqr + __popcll(eqb & lt) < take_eq)))));
      eqr += __popcll(eqb);
      sb[u] = __ballot(sel);
    }
    return run;
  };
  for (int i0 = 0, run = rank_base, eqr = eq_base; i0 < R; i0 += kGrp) {
    unsigned long long sb[kGrp];
    run = select_group(i0, run, eqr, sb);
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      wsel += __popcll(sb[u]);
      if (i0 + u < 64 && ((sb[u] >> lane) & 1ull)) sbits |= 1ull << (i0 + u);
    }
  }
  int sel_tot;
  const int out_base = wave_scan(wsel, wt_sel, &sel_tot) + out0;
  if (wsel == 0 && !want_slots) return;
  // In place, every member row also records the slot that reads it (-1:
  // dropped), for the ordering of the in-place gather.
  int* so = want_slots ? slot_of + off : nullptr;
  const int heads = SHARED ? dm.Hkv : 1;
  for (int i0 = 0, run = rank_base, eqr = eq_base, o = out_base; i0 < R; i0 += kGrp) {
    unsigned long long sb[kGrp];
    if (bits_ok) {
#pragma unroll
      for (int u = 0; u < kGrp; ++u) sb[u] = __ballot(((sbits >> min(i0 + u, 63)) & 1ull) && i0 + u < R);
    } else {
      run = select_group(i0, run, eqr, sb);
    }
#pragma unroll
    for (int u = 0; u < kGrp; ++u) {
      const int row = wrow0 + (i0 + u) * 64 + lane;
      if ((sb[u] >> lane) & 1ull) {
        const int slot = o + __popcll(sb[u] & lt);
        for (int h = 0; h < heads; ++h) {
          ig[(int64_t)h * dm.max_tokens + slot] = row;
          if (so) so[(int64_t)h * dm.max_tokens + row] = slot;
        }
      } else if (so && i0 + u < R && row < N && member_at(i0 + u, row)) {
        for (int h = 0; h < heads; ++h) so[(int64_t)h * dm.max_tokens + row] = -1;
      }
      o += __popcll(sb[u]);
    }
  }
}

// psi_topk for working sets of at most kRegRows rows: each lane keeps the
// keys of its rows (wave w owns rows 512 w .. 512 w + 511, step i the 64
// rows from 512 w + 64 i) in registers from the one round of reads to the
// emission.  The radix select runs on them directly, 12-bit digits below
// the bits all keys share, two LDS histograms taking turns (one is cleared
// while the other is scanned), and stops at the first digit whose bin is
// kept whole.
constexpr int kRegSteps = 8;
constexpr int kRegRows = kRegSteps * kSelThreads;

template <bool SHARED>
__global__ __launch_bounds__(kSelThreads) void psi_topk_reg(const LayerDesc* __restrict__ layers, Dims dm, float lambda,
                                                            const float* __restrict__ a, const float* __restrict__ s,
                                                            const int32_t* __restrict__ budgets,
                                                            int32_t* __restrict__ idx, int* __restrict__ eff,
                                                            int* __restrict__ slot_of, int* __restrict__ ctl) {
  __shared__ int hist[2][kBins];
  __shared__ int wsum[1][kSelWaves];
  __shared__ int s_bin, s_need, s_cnt, s_lcnt;
  __shared__ uint32_t s_thr;
  __shared__ int wt_mem[kSelWaves], wt_eq[kSelWaves], wt_sel[kSelWaves];
  __shared__ uint32_t wmin[kSelWaves], wmax[kSelWaves];
  const int mu = blockIdx.x, g = blockIdx.y, l = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int64_t off = ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const float* ag = a + (SHARED ? (int64_t)l * dm.max_tokens : off);
  const float* sg = s + (SHARED ? (int64_t)l * dm.max_tokens : off);
  const int row0 = wave * 64 * kRegSteps + lane;
  // a, s and the budgets are requested before the layer's descriptor arrives
  // (indices kept inside the buffers' rows; rows past N are not used)
  float av[kRegSteps], sv[kRegSteps];
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) {
    const int j = min(row0 + 64 * i, (int)dm.max_tokens - 1);
    av[i] = gload<float>(ag + j);
    sv[i] = gload<float>(sg + j);
  }
  const int bud_mu = budgets[2 * l + mu], bud_v = budgets[2 * l];
  if (ctl != nullptr && blockIdx.x == 0 && g == 0 && l == 0 && threadIdx.x == 0)
    ctl[1] = 0;  // staging rows needed beyond the reserve, this call
  const LayerDesc& Ld = layers[l];
  const int N = Ld.n;
  const uint8_t* mod = Ld.mod;
  const int cap = Ld.out_cap;
  int mv[kRegSteps];
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) mv[i] = gload<uint8_t>(mod + max(0, min(row0 + 64 * i, N - 1)));
  for (int i = threadIdx.x; i < kBins; i += kSelThreads) hist[0][i] = 0;
  if (threadIdx.x == 0) s_lcnt = 0;
  // keys of the member rows, their count and range
  bool mb[kRegSteps];
  uint32_t kk[kRegSteps];
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
  int wcount = 0;
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) {
    mb[i] = (row0 + 64 * i < N) & ((mv[i] ? 1 : 0) == mu);
    kk[i] = psi_key(av[i], sv[i], lambda);
    wcount += __popcll(__ballot(mb[i]));
    kmin = mb[i] ? min(kmin, kk[i]) : kmin;
    kmax = mb[i] ? max(kmax, kk[i]) : kmax;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
  }
  if (lane == 0) { wt_mem[wave] = wcount; wmin[wave] = kmin; wmax[wave] = kmax; }
  __syncthreads();  // counts and ranges of the waves; histogram 0 cleared
  int K = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    K += wt_mem[w];
    kmin = min(kmin, wmin[w]);
    kmax = max(kmax, wmax[w]);
  }
  K = uniform(K);
  kmin = (uint32_t)uniform((int)kmin);
  kmax = (uint32_t)uniform((int)kmax);
  // Budgets as applied: each modality's within its rows, visual first
  // within the output capacity, audio in what remains.
  const int Kv = mu ? N - K : K;
  const int Mv = min(min(max(bud_v, 0), Kv), cap);
  const int M = mu ? min(min(max(bud_mu, 0), K), cap - Mv) : Mv;
  if (g == 0 && threadIdx.x == 0) eff[2 * l + mu] = M;
  const int out0 = mu ? Mv : 0;
  const bool all = M >= K, pick = !all && M > 0;

  // Radix select of the M-th largest key: keep the keys above thr and the
  // first take_eq keys equal to it.
  uint32_t thr = 0;
  int take_eq = 0, n_eq = 0;
  if (pick) {
    const int width = (kmin ^ kmax) ? 32 - __clz(kmin ^ kmax) : 0;  // low bits in which keys differ
    const uint32_t low = width < 32 ? (1u << width) - 1u : 0xFFFFFFFFu;
    uint32_t prefix = kmin & ~low, mask = ~low;
    int need = M, cnt = K, buf = 0;
    bool whole = false, ranked = false;
    for (int top = width; top > 0 && !whole;) {
      const int shift = max(0, top - kDigit);
      const uint32_t dmask = (1u << (top - shift)) - 1u;
#pragma unroll
      for (int i = 0; i < kRegSteps; ++i)
        if (mb[i] && (kk[i] & mask) == prefix) atomicAdd(&hist[buf][(kk[i] >> shift) & dmask], 1);
      __syncthreads();
      // bins from the top: thread t holds bins btop - q, q < PER; the other
      // histogram is cleared for the next digit meanwhile
      constexpr int PER = kBins / kSelThreads;
      const int btop = kBins - 1 - PER * (int)threadIdx.x;
      int h[PER], mine = 0;
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        h[q] = hist[buf][btop - q];
        hist[buf ^ 1][btop - q] = 0;
        mine += h[q];
      }
      int v[1] = {mine}, tot[1];
      block_inclusive<1>(v, wsum, tot);
      const int above = v[0] - mine;
      int bi, need_in, cnt_in;
      crossing_bin<PER>(h, above, need, bi, need_in, cnt_in);
      if (above < need && need <= above + mine) { s_bin = btop - bi; s_need = need_in; s_cnt = cnt_in; }
      __syncthreads();
      prefix |= (uint32_t)uniform(s_bin) << shift;
      mask |= dmask << shift;
      need = uniform(s_need);
      cnt = uniform(s_cnt);
      whole = need >= cnt;
      top = shift;
      buf ^= 1;
      __syncthreads();  // every thread has read s_bin, s_need, s_cnt
      if (!whole && top > 0 && cnt <= kListMax) {
        // Few keys left in the threshold's bin: collect them into the next
        // digit's (unused) histogram and rank each against the others, four
        // threads per key, instead of further digits.  The key with fewer
        // than `need` keys strictly above it and at least `need` counting
        // its equals is the threshold.
        int* cand = hist[buf];
#pragma unroll
        for (int i = 0; i < kRegSteps; ++i) {
          const bool m = mb[i] & ((kk[i] & mask) == prefix);
          const unsigned long long b = __ballot(m);
          int base = 0;
          if (lane == 0 && b) base = atomicAdd(&s_lcnt, __popcll(b));
          base = __shfl(base, 0, 64);
          if (m) cand[base + __popcll(b & lt)] = (int)kk[i];
        }
        __syncthreads();
        static_assert(4 * kListMax <= kSelThreads, "four threads per candidate");
        const int ci = (int)threadIdx.x >> 2, part = (int)threadIdx.x & 3;
        const uint32_t c = ci < cnt ? (uint32_t)cand[ci] : 0u;
        int gt = 0, eq = 0;
        for (int u = part; u < cnt; u += 4) {
          const uint32_t x = (uint32_t)cand[u];
          gt += x > c ? 1 : 0;
          eq += x == c ? 1 : 0;
        }
        gt += __shfl_xor(gt, 1, 64);
        eq += __shfl_xor(eq, 1, 64);
        gt += __shfl_xor(gt, 2, 64);
        eq += __shfl_xor(eq, 2, 64);
        // every candidate equal to the threshold writes the same values
        if (ci < cnt && part == 0 && gt < need && need <= gt + eq) { s_thr = c; s_need = need - gt; s_cnt = eq; }
        __syncthreads();
        thr = (uint32_t)uniform((int)s_thr);
        take_eq = uniform(s_need);
        n_eq = uniform(s_cnt);
        ranked = true;
        break;
      }
    }
    if (ranked) {
      // thr, take_eq and n_eq set by the ranking
    } else if (whole) {
      thr = prefix - 1u;  // the keys from prefix up: the whole bin and every bin above it
    } else {
      thr = prefix;       // every bit resolved: the threshold key itself
      take_eq = need;
      n_eq = cnt;
    }
  }

  // Ordered emission: rows above thr and the first take_eq rows equal to it
  // (ties to the lower row), in ascending row order.
  const bool eq_ranks = pick && take_eq > 0 && take_eq < n_eq;
  bool keep_eq[kRegSteps];
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) keep_eq[i] = take_eq > 0;
  if (eq_ranks) {
    unsigned long long eb[kRegSteps];
    int weq = 0;
#pragma unroll
    for (int i = 0; i < kRegSteps; ++i) {
      eb[i] = __ballot(mb[i] & (kk[i] == thr));
      weq += __popcll(eb[i]);
    }
    int eq_tot;
    int run = wave_scan(weq, wt_eq, &eq_tot);
#pragma unroll
    for (int i = 0; i < kRegSteps; ++i) {
      if ((eb[i] >> lane) & 1ull) keep_eq[i] = run + __popcll(eb[i] & lt) < take_eq;
      run += __popcll(eb[i]);
    }
  }
  unsigned long long sb[kRegSteps];
  int wsel = 0;
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) {
    const bool sel = mb[i] & (all | (pick & ((kk[i] > thr) | ((kk[i] == thr) & keep_eq[i]))));
    sb[i] = __ballot(sel);
    wsel += __popcll(sb[i]);
  }
  int sel_tot;
  int o = wave_scan(wsel, wt_sel, &sel_tot) + out0;
  const bool want_slots = Ld.inplace != 0 && slot_of != nullptr;
  int32_t* ig = idx + off;
  int* so = want_slots ? slot_of + off : nullptr;
  const int heads = SHARED ? dm.Hkv : 1;
#pragma unroll
  for (int i = 0; i < kRegSteps; ++i) {
    const int row = row0 + 64 * i;
    if ((sb[i] >> lane) & 1ull) {
      const int slot = o + __popcll(sb[i] & lt);
      for (int h = 0; h < heads; ++h) {
        ig[(int64_t)h * dm.max_tokens + slot] = row;
        if (so) so[(int64_t)h * dm.max_tokens + row] = slot;
      }
    } else if (so && mb[i]) {
      for (int h = 0; h < heads; ++h) so[(int64_t)h * dm.max_tokens + row] = -1;
    }
    o += __popcll(sb[i]);
  }
}

// ---------------------------------------------------------------------------
// Top-k split over several workgroups per (layer, KV head), for long working
// sets.  A row's key is psi's order-preserving bits with its modality in bit
// 31.  The M-th largest key of a modality is located by its first 12-bit
// digit (key bits 30..19) in a histogram summed over the whole working set,
// then among the keys in that bin (the "candidates", a small share of the
// rows unless psi piles up in one narrow range) by the remaining 19 bits.
//   topk_hist  4096 rows per workgroup: keys to `keys`; first-digit
//              histograms of both modalities in LDS, added into the (layer,
//              KV head)'s histograms in global memory.
//   topk_bin   2048-row slices: every workgroup scans the histograms for the
//              budgets as applied and each modality's threshold bin, counts
//              its slice's keys above that bin (every member when all are
//              kept) and writes the keys in it, in row order, to the slice's
//              region of `cand` (visual from the front, audio from the back).
//   topk_emit  per slice: the candidates of all slices, ranked in LDS by the
//              two remaining digits, give the exact threshold key and how
//              many keys equal to it are kept (the first ones in row order);
//              the kept rows in front of the slice are counted and the
//              slice's kept rows written in ascending order.  It also clears
//              the histograms, which topk_bin has finished reading.
// ---------------------------------------------------------------------------
constexpr int kTkThreads = 1024;
constexpr int kTkWaves = kTkThreads / 64;
static_assert(kTkWaves == kSelWaves, "the scans are sized for one workgroup size");
constexpr int kHistRows = 4096;                       // rows per topk_hist workgroup
constexpr int kSliceSteps = kTopkSlice / kTkThreads;  // rows per lane of a slice
constexpr int kCandLds = 4096;                        // candidates of a modality ranked in LDS
constexpr int kShift1 = 19, kShift2 = 7;              // digits: key bits 30..19, 18..7, 6..0
constexpr uint32_t kKeyBits = 0x7FFFFFFFu;
static_assert(kTopkBins % (4 * kTkThreads) == 0 && kTopkSlice % kTkThreads == 0, "whole bins and rows per lane");
static_assert(kTopkMaxSlices <= kTkThreads && (2 << kShift2) <= kTkThreads, "one slice and one bin per thread");

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
__device__ inline uint2 gload8(const void* p) {
  const u32x2 v = gload<u32x2>(p);
  return make_uint2(v[0], v[1]);
}

template <bool SHARED>
__global__ __launch_bounds__(kTkThreads) void topk_hist(const LayerDesc* __restrict__ layers, Dims dm, float lambda,
                                                         const float* __restrict__ a, const float* __restrict__ s,
                                                         uint32_t* __restrict__ keys, int* __restrict__ hist,
                                                         int* __restrict__ ccount, int* __restrict__ ctl) {
  __shared__ int h[2 * kTopkBins];
  const int l = blockIdx.z, g = blockIdx.y, r0 = blockIdx.x * kHistRows;
  const int64_t unit = (int64_t)l * dm.Hkv + g;
  const int64_t in_off = SHARED ? (int64_t)l * dm.max_tokens : unit * dm.max_tokens;
  const float* ag = a + in_off;
  const float* sg = s + in_off;
  constexpr int R = kHistRows / kTkThreads;
  // a and s are requested before the layer's descriptor arrives (indices
  // kept inside the buffers' rows; rows past N are not used)
  float av[R], sv[R];
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int j = min(r0 + u * kTkThreads + (int)threadIdx.x, (int)dm.max_tokens - 1);
    av[u] = gload<float>(ag + j);
    sv[u] = gload<float>(sg + j);
  }
  if (ctl != nullptr && blockIdx.x == 0 && g == 0 && l == 0 && threadIdx.x == 0)
    ctl[1] = 0;  // staging rows needed beyond the reserve, this call
  if (blockIdx.x == 0 && threadIdx.x < 2) ccount[unit * 2 + threadIdx.x] = 0;  // topk_bin lists after this kernel
  const int N = layers[l].n;
  if (r0 >= N) return;
  const uint8_t* mod = layers[l].mod;
  uint32_t* kg = keys + unit * topk_stride(dm.max_tokens);
  int* gh = hist + unit * 2 * kTopkBins;
  int mv[R];
#pragma unroll
  for (int u = 0; u < R; ++u) mv[u] = gload<uint8_t>(mod + min(r0 + u * kTkThreads + (int)threadIdx.x, N - 1));
  int4* h4 = reinterpret_cast<int4*>(h);
  for (int i = threadIdx.x; i < 2 * kTopkBins / 4; i += kTkThreads) h4[i] = make_int4(0, 0, 0, 0);
  __syncthreads();  // histograms cleared
#pragma unroll
  for (int u = 0; u < R; ++u) {
    const int j = r0 + u * kTkThreads + (int)threadIdx.x;
    if (j < N) {
      const uint32_t key = psi_key(av[u], sv[u], lambda);
      const uint32_t mu = mv[u] ? 1u : 0u;
      kg[j] = key | (mu << 31);
      atomicAdd(&h[mu * kTopkBins + (key >> kShift1)], 1);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 2 * kTopkBins / 4; i += kTkThreads) {
    const int4 c = h4[i];
    if (c.x) atomicAdd(gh + 4 * i, c.x);
    if (c.y) atomicAdd(gh + 4 * i + 1, c.y);
    if (c.z) atomicAdd(gh + 4 * i + 2, c.z);
    if (c.w) atomicAdd(gh + 4 * i + 3, c.w);
  }
}

// Segment record (tk_seg), per (layer, KV head, modality).
enum { SEG_MODE, SEG_BIN, SEG_NEED, SEG_CNT, SEG_M, SEG_OUT0, SEG_K };
enum { MODE_NONE = 0, MODE_ALL = 1, MODE_PICK = 2 };

template <bool SHARED>
__global__ __launch_bounds__(kTkThreads) void topk_bin(const LayerDesc* __restrict__ layers, Dims dm,
                                                        const uint32_t* __restrict__ keys, const int* __restrict__ hist,
                                                        const int32_t* __restrict__ budgets, int* __restrict__ seg,
                                                        int* __restrict__ slice, uint2* __restrict__ cand,
                                                        int* __restrict__ ccount, int* __restrict__ eff) {
  __shared__ int wsum[2][kTkWaves];
  __shared__ int s_bin[2], s_need[2], s_cnt[2], s_base[2];
  __shared__ int wc[2][kSliceSteps][kTkWaves];  // candidates per (modality, step, wave)
  __shared__ int wa[2][kTkWaves];               // keys above the bin per (modality, wave)
  const int l = blockIdx.z, g = blockIdx.y, p = blockIdx.x;
  const int r0 = p * kTopkSlice;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int64_t unit = (int64_t)l * dm.Hkv + g;
  const int64_t stride = topk_stride(dm.max_tokens);
  const uint32_t* kg = keys + unit * stride;
  // Reads that need no descriptor first: the histograms (bins highest first:
  // thread t holds bins btop - i, i < PER, of each modality) and the slice's
  // keys (whole slices lie inside the key buffer; rows past N are not used).
  constexpr int PER = kTopkBins / kTkThreads;
  const int btop = kTopkBins - 1 - PER * (int)threadIdx.x;
  int hb[2][PER];
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
      const uint4 v = gload16(hist + unit * 2 * kTopkBins + mu * kTopkBins + btop - (PER - 1) + 4 * q);
      hb[mu][PER - 1 - 4 * q] = (int)v.x;
      hb[mu][PER - 2 - 4 * q] = (int)v.y;
      hb[mu][PER - 3 - 4 * q] = (int)v.z;
      hb[mu][PER - 4 - 4 * q] = (int)v.w;
    }
  }
  uint32_t kk[kSliceSteps];
#pragma unroll
  for (int u = 0; u < kSliceSteps; ++u) kk[u] = gload<uint32_t>(kg + r0 + u * kTkThreads + (int)threadIdx.x);
  const int bud_v = budgets[2 * l], bud_a = budgets[2 * l + 1];
  const int N = layers[l].n;
  if (r0 >= N && p > 0) return;  // slice 0 always writes the segment records
  const int cap = layers[l].out_cap;
  int mine[2] = {0, 0};
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    mine[0] += hb[0][i];
    mine[1] += hb[1][i];
  }
  int incl[2] = {mine[0], mine[1]}, K[2];
  block_inclusive<2>(incl, wsum, K);
  // budgets as applied: each modality's within its rows, visual first within the output capacity
  int M[2];
  M[0] = min(min(max(bud_v, 0), K[0]), cap);
  M[1] = min(min(max(bud_a, 0), K[1]), cap - M[0]);
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    const int above = incl[mu] - mine[mu];
    const int m = M[mu];
    int i, need_in, cnt;
    crossing_bin<PER>(hb[mu], above, m, i, need_in, cnt);
    if (0 < m && m < K[mu] && above < m && m <= above + mine[mu]) { s_bin[mu] = btop - i; s_need[mu] = need_in; s_cnt[mu] = cnt; }
  }
  __syncthreads();
  // (the same in every lane: kept in scalar registers, so that the flags
  // below are plain lane arithmetic)
  int mode[2], b1[2];
  bool whole[2];  // the threshold's whole first-digit bin is kept: no candidates
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    M[mu] = uniform(M[mu]);
    K[mu] = uniform(K[mu]);
    mode[mu] = M[mu] == 0 ? MODE_NONE : M[mu] >= K[mu] ? MODE_ALL : MODE_PICK;
    b1[mu] = mode[mu] == MODE_PICK ? uniform(s_bin[mu]) : 0;
    whole[mu] = mode[mu] == MODE_PICK && uniform(s_need[mu]) >= uniform(s_cnt[mu]);
  }
  if (p == 0 && threadIdx.x < 2) {
    const int mu = threadIdx.x;
    int* sr = seg + (unit * 2 + mu) * 8;
    sr[SEG_MODE] = mode[mu];
    sr[SEG_BIN] = b1[mu];
    sr[SEG_NEED] = mode[mu] == MODE_PICK ? s_need[mu] : 0;
    sr[SEG_CNT] = mode[mu] == MODE_PICK ? s_cnt[mu] : 0;
    sr[SEG_M] = M[mu];
    sr[SEG_OUT0] = mu ? M[0] : 0;
    sr[SEG_K] = K[mu];
    if (g == 0) eff[2 * l + mu] = M[mu];
  }
  if (r0 >= N) return;
  int na[2] = {0, 0};
  unsigned long long cb[2][kSliceSteps];
#pragma unroll
  for (int u = 0; u < kSliceSteps; ++u) {
    const bool valid = r0 + u * kTkThreads + (int)threadIdx.x < N;
    const int mu_u = (int)(kk[u] >> 31);
    const int d1 = (int)((kk[u] & kKeyBits) >> kShift1);
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      const bool m = valid & (mu_u == mu);
      const bool all = mode[mu] == MODE_ALL, pick = mode[mu] == MODE_PICK;
      const bool above_f = m & (all | (pick & ((d1 > b1[mu]) | (whole[mu] & (d1 == b1[mu])))));
      const bool cand_f = m & pick & !whole[mu] & (d1 == b1[mu]);
      na[mu] += __popcll(__ballot(above_f));
      cb[mu][u] = __ballot(cand_f);
      if (lane == 0) wc[mu][u][wave] = __popcll(cb[mu][u]);
    }
  }
  if (lane == 0) { wa[0][wave] = na[0]; wa[1][wave] = na[1]; }
  __syncthreads();
  // The slice's count above the bin, and room for its candidates in the
  // (layer, KV head)'s list (one atomic per modality).
  if (threadIdx.x < 2) {
    const int mu = threadIdx.x;
    int above = 0, n = 0;
#pragma unroll
    for (int w = 0; w < kTkWaves; ++w) {
      above += wa[mu][w];
#pragma unroll
      for (int u = 0; u < kSliceSteps; ++u) n += wc[mu][u][w];
    }
    slice[(unit * kTopkMaxSlices + p) * 2 + mu] = above;
    s_base[mu] = n ? atomicAdd(ccount + unit * 2 + mu, n) : 0;
  }
  __syncthreads();
  uint2* cl = cand + unit * stride;
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    int run = s_base[mu];
#pragma unroll
    for (int u = 0; u < kSliceSteps; ++u) {
      int before = run, all = 0;
#pragma unroll
      for (int w = 0; w < kTkWaves; ++w) {
        const int c = wc[mu][u][w];
        before += w < wave ? c : 0;
        all += c;
      }
      if ((cb[mu][u] >> lane) & 1ull) {
        const int r = before + __popcll(cb[mu][u] & lt);
        cl[mu ? stride - 1 - r : r] = make_uint2(kk[u] & kKeyBits, (uint32_t)(r0 + u * kTkThreads + (int)threadIdx.x));
      }
      run += all;
    }
  }
}

template <bool SHARED>
__global__ __launch_bounds__(kTkThreads) void topk_emit(const LayerDesc* __restrict__ layers, Dims dm,
                                                         const uint32_t* __restrict__ keys, int* __restrict__ hist,
                                                         const int* __restrict__ seg, const int* __restrict__ slice,
                                                         const uint2* __restrict__ cand, int32_t* __restrict__ idx,
                                                         int* __restrict__ slot_of) {
  __shared__ uint32_t ck[2][kCandLds];            // candidate keys of each modality; bit 31: row in front of the slice
  __shared__ int hb[2][kTopkBins];                // digit histograms
  __shared__ int apre[2][kTopkMaxSlices + 1];     // keys above the first-digit bin in front of slice i
  __shared__ int wsum0[2][kTkWaves], wsum1[2][kTkWaves], wsum2[2][kTkWaves], wsum3[4][kTkWaves];
  __shared__ int s_bin[2], s_need[2], s_cnt[2];
  __shared__ int wc[2][kSliceSteps][kTkWaves];
  const int l = blockIdx.z, g = blockIdx.y, p = blockIdx.x;
  const int r0 = p * kTopkSlice;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int64_t unit = (int64_t)l * dm.Hkv + g;
  const int64_t stride = topk_stride(dm.max_tokens);
  const uint32_t* kg = keys + unit * stride;
  const uint2* cl = cand + unit * stride;

  // Reads that need no descriptor first: the slice's keys, the slice table
  // (thread t: slice t) and the segment records.
  uint32_t kk[kSliceSteps];
#pragma unroll
  for (int u = 0; u < kSliceSteps; ++u) kk[u] = gload<uint32_t>(kg + r0 + u * kTkThreads + (int)threadIdx.x);
  uint2 st = make_uint2(0, 0);
  if (threadIdx.x < gridDim.x) st = gload8(slice + (unit * kTopkMaxSlices + threadIdx.x) * 2);
  int sr[2][7];
#pragma unroll
  for (int mu = 0; mu < 2; ++mu)
#pragma unroll
    for (int f = 0; f < 7; ++f) sr[mu][f] = uniform(seg[(unit * 2 + mu) * 8 + f]);
  const LayerDesc& Ld = layers[l];
  const int N = Ld.n;
  if (r0 >= N) return;
  const int P = (N + kTopkSlice - 1) / kTopkSlice;
  if ((int)threadIdx.x >= P) st = make_uint2(0, 0);
  // This slice's share of the histograms back to zero for the next call.
  {
    constexpr int V4 = 2 * kTopkBins / 4;
    const int per = (V4 + P - 1) / P;
    int4* h4 = reinterpret_cast<int4*>(hist + unit * 2 * kTopkBins);
    for (int i = p * per + (int)threadIdx.x; i < min(V4, (p + 1) * per); i += kTkThreads) h4[i] = make_int4(0, 0, 0, 0);
  }
  // Keys above the first-digit bin in front of each slice.
  {
    int v[2] = {(int)st.x, (int)st.y}, tot[2];
    block_inclusive<2>(v, wsum0, tot);
    if ((int)threadIdx.x < P) {
      apre[0][threadIdx.x + 1] = v[0];
      apre[1][threadIdx.x + 1] = v[1];
    }
    if (threadIdx.x == 0) { apre[0][0] = 0; apre[1][0] = 0; }
    __syncthreads();
  }

  // Exact threshold of each modality that ranks: keep the keys above thr
  // and the first `take` keys equal to it.  Both modalities go through each
  // phase together.
  uint32_t thr[2] = {0u, 0u}, b1[2];
  int take[2] = {0, 0}, n_eq[2] = {0, 0}, gtb[2], eqb[2] = {0, 0}, need1[2], C[2];
  bool rank[2], whole[2], in_lds[2];
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    b1[mu] = (uint32_t)sr[mu][SEG_BIN];
    need1[mu] = sr[mu][SEG_NEED];
    C[mu] = sr[mu][SEG_CNT];  // the keys in the first-digit bin: the listed candidates
    gtb[mu] = apre[mu][p];
    rank[mu] = sr[mu][SEG_MODE] == MODE_PICK && need1[mu] < C[mu];
    whole[mu] = sr[mu][SEG_MODE] == MODE_PICK && !rank[mu];  // the whole first-digit bin is kept
    in_lds[mu] = C[mu] <= kCandLds;
    if (whole[mu]) thr[mu] = (b1[mu] << kShift1) - 1u;  // counted above the bin by topk_bin
  }
  if (rank[0] || rank[1]) {
    // candidate i of modality mu as its key with bit 31 set when its row is
    // in front of this slice
    auto cand_at = [&](int mu, int i) {
      const uint2 c = gload8(cl + (mu ? stride - 1 - i : i));
      return c.x | (c.y < (uint32_t)r0 ? 0x80000000u : 0u);
    };
    // visit(key) over candidates [0, n) of modality mu, eight per lane in flight
    auto for_cands = [&](int mu, int n, auto&& visit) {
      for (int i0 = 0; i0 < n; i0 += 8 * kTkThreads) {
        uint32_t v[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = i0 + b * kTkThreads + (int)threadIdx.x;
          v[b] = i < n ? (in_lds[mu] ? ck[mu][i] : cand_at(mu, i)) : 0u;
        }
#pragma unroll
        for (int b = 0; b < 8; ++b)
          if (i0 + b * kTkThreads + (int)threadIdx.x < n) visit(v[b]);
      }
    };
    {
      int4* h4 = reinterpret_cast<int4*>(&hb[0][0]);
      for (int i = threadIdx.x; i < 2 * kTopkBins / 4; i += kTkThreads) h4[i] = make_int4(0, 0, 0, 0);
    }
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      if (!rank[mu] || !in_lds[mu]) continue;
      for (int i0 = 0; i0 < C[mu]; i0 += 8 * kTkThreads) {
        uint32_t v[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = i0 + b * kTkThreads + (int)threadIdx.x;
          v[b] = i < C[mu] ? cand_at(mu, i) : 0u;
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
          const int i = i0 + b * kTkThreads + (int)threadIdx.x;
          if (i < C[mu]) ck[mu][i] = v[b];
        }
      }
    }
    __syncthreads();  // histograms cleared, candidates in LDS
    // second digit (key bits 18..7)
#pragma unroll
    for (int mu = 0; mu < 2; ++mu)
      if (rank[mu]) for_cands(mu, C[mu], [&](uint32_t key) { atomicAdd(&hb[mu][(key >> kShift2) & (kTopkBins - 1)], 1); });
    __syncthreads();
    {
      constexpr int PER = kTopkBins / kTkThreads;
      const int btop = kTopkBins - 1 - PER * (int)threadIdx.x;
      int h[2][PER], mine[2] = {0, 0};
#pragma unroll
      for (int mu = 0; mu < 2; ++mu)
#pragma unroll
        for (int i = 0; i < PER; ++i) { h[mu][i] = hb[mu][btop - i]; mine[mu] += h[mu][i]; }
      int v[2] = {mine[0], mine[1]}, tot[2];
      block_inclusive<2>(v, wsum1, tot);
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const int above = v[mu] - mine[mu];
        const int need = need1[mu];
        int i, need_in, cnt;
        crossing_bin<PER>(h[mu], above, need, i, need_in, cnt);
        if (rank[mu] && above < need && need <= above + mine[mu]) { s_bin[mu] = btop - i; s_need[mu] = need_in; s_cnt[mu] = cnt; }
      }
      __syncthreads();
    }
    uint32_t pre2[2];
    int need2[2];
    bool third[2];
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      pre2[mu] = (b1[mu] << (kShift1 - kShift2)) | (uint32_t)uniform(s_bin[mu]);  // key bits 30..7
      need2[mu] = uniform(s_need[mu]);
      third[mu] = rank[mu] && need2[mu] < uniform(s_cnt[mu]);
      if (rank[mu] && !third[mu]) thr[mu] = (pre2[mu] << kShift2) - 1u;  // the whole second-digit bin is kept
    }
    if (third[0] || third[1]) {
      __syncthreads();  // every thread has read the histograms and s_bin, s_need, s_cnt
      if (threadIdx.x < 2u << kShift2) hb[threadIdx.x >> kShift2][threadIdx.x & ((1u << kShift2) - 1u)] = 0;
      __syncthreads();
#pragma unroll
      for (int mu = 0; mu < 2; ++mu)
        if (third[mu])
          for_cands(mu, C[mu], [&](uint32_t key) {
            if (((key & kKeyBits) >> kShift2) == pre2[mu]) atomicAdd(&hb[mu][key & ((1u << kShift2) - 1u)], 1);
          });
      __syncthreads();
      const int t = (int)threadIdx.x;
      const int bin = (1 << kShift2) - 1 - t;
      int c[2], v[2], tot[2];
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) c[mu] = v[mu] = t < (1 << kShift2) ? hb[mu][bin] : 0;
      block_inclusive<2>(v, wsum2, tot);
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        const int above = v[mu] - c[mu];
        if (third[mu] && c[mu] > 0 && above < need2[mu] && need2[mu] <= above + c[mu]) {
          s_bin[mu] = bin; s_need[mu] = need2[mu] - above; s_cnt[mu] = c[mu];
        }
      }
      __syncthreads();
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        if (!third[mu]) continue;
        thr[mu] = (pre2[mu] << kShift2) | (uint32_t)uniform(s_bin[mu]);
        take[mu] = uniform(s_need[mu]);
        n_eq[mu] = uniform(s_cnt[mu]);
      }
    }
    // kept candidates of the slices in front: above thr, or equal to it
    int v[4] = {0, 0, 0, 0}, tot[4];
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      if (!rank[mu]) continue;
      const uint32_t th = thr[mu];
      int gt = 0, eq = 0;
      for_cands(mu, C[mu], [&](uint32_t key) {
        const bool front = (key >> 31) != 0;
        key &= kKeyBits;
        gt += front && key > th ? 1 : 0;
        eq += front && key == th ? 1 : 0;
      });
      v[2 * mu] = gt;
      v[2 * mu + 1] = eq;
    }
    block_inclusive<4>(v, wsum3, tot);
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      if (!rank[mu]) continue;
      gtb[mu] += tot[2 * mu];
      eqb[mu] = tot[2 * mu + 1];
    }
  }

  // Emission: the slice's kept rows in ascending order.
  const bool need_rank[2] = {rank[0] && take[0] > 0 && take[0] < n_eq[0], rank[1] && take[1] > 0 && take[1] < n_eq[1]};
  bool keep_eq[kSliceSteps];
#pragma unroll
  for (int u = 0; u < kSliceSteps; ++u) keep_eq[u] = true;
  if (need_rank[0] || need_rank[1]) {  // ranks among the keys equal to a threshold
    unsigned long long eb[2][kSliceSteps];
#pragma unroll
    for (int u = 0; u < kSliceSteps; ++u) {
      const bool valid = r0 + u * kTkThreads + (int)threadIdx.x < N;
      const int mu_u = (int)(kk[u] >> 31);
      const uint32_t k = kk[u] & kKeyBits;
#pragma unroll
      for (int mu = 0; mu < 2; ++mu) {
        eb[mu][u] = __ballot(valid & (mu_u == mu) & need_rank[mu] & (k == thr[mu]));
        if (lane == 0) wc[mu][u][wave] = __popcll(eb[mu][u]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      int run = 0;
#pragma unroll
      for (int u = 0; u < kSliceSteps; ++u) {
        int before = run, all = 0;
#pragma unroll
        for (int w = 0; w < kTkWaves; ++w) {
          const int c = wc[mu][u][w];
          before += w < wave ? c : 0;
          all += c;
        }
        if ((eb[mu][u] >> lane) & 1ull) keep_eq[u] = eqb[mu] + before + __popcll(eb[mu][u] & lt) < take[mu];
        run += all;
      }
    }
    __syncthreads();  // before wc is reused
  }
  unsigned long long sb[2][kSliceSteps];
#pragma unroll
  for (int u = 0; u < kSliceSteps; ++u) {
    const bool valid = r0 + u * kTkThreads + (int)threadIdx.x < N;
    const int mu_u = (int)(kk[u] >> 31);
    const uint32_t k = kk[u] & kKeyBits;
#pragma unroll
    for (int mu = 0; mu < 2; ++mu) {
      const bool all = sr[mu][SEG_MODE] == MODE_ALL, pick = sr[mu][SEG_MODE] == MODE_PICK;
      const bool sel = valid & (mu_u == mu) & (all | (pick & ((k > thr[mu]) | ((k == thr[mu]) & (take[mu] > 0) & keep_eq[u]))));
      sb[mu][u] = __ballot(sel);
      if (lane == 0) wc[mu][u][wave] = __popcll(sb[mu][u]);
    }
  }
  __syncthreads();
  const bool want_slots = Ld.inplace != 0 && slot_of != nullptr;
  const int heads = SHARED ? dm.Hkv : 1;
  int32_t* ig = idx + unit * dm.max_tokens;
  int* so = want_slots ? slot_of + unit * dm.max_tokens : nullptr;
#pragma unroll
  for (int mu = 0; mu < 2; ++mu) {
    int run = sr[mu][SEG_OUT0] + gtb[mu] + min(eqb[mu], take[mu]);
#pragma unroll
    for (int u = 0; u < kSliceSteps; ++u) {
      int before = run, all = 0;
#pragma unroll
      for (int w = 0; w < kTkWaves; ++w) {
        const int c = wc[mu][u][w];
        before += w < wave ? c : 0;
        all += c;
      }
      const int row = r0 + u * kTkThreads + (int)threadIdx.x;
      if ((sb[mu][u] >> lane) & 1ull) {
        const int slot = before + __popcll(sb[mu][u] & lt);
        for (int h = 0; h < heads; ++h) {
          ig[(int64_t)h * dm.max_tokens + slot] = row;
          if (so) so[(int64_t)h * dm.max_tokens + row] = slot;
        }
      } else if (so && row < N && (int)(kk[u] >> 31) == mu) {
        for (int h = 0; h < heads; ++h) so[(int64_t)h * dm.max_tokens + row] = -1;
      }
      run += all;
    }
  }
}

constexpr int kCompactRows = 32;  // output rows per workgroup of the out-of-place gather

template <typename T, int D>
__global__ __launch_bounds__(256) void gather_compact(const LayerDesc* __restrict__ layers, Dims dm,
                                                      const int32_t* __restrict__ idx, const int* __restrict__ eff,
                                                      const int* __restrict__ ctl) {
  constexpr int CPR = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  constexpr int RPP = 256 / CPR;                // rows per pass
  constexpr int ROWS = kCompactRows;            // rows per workgroup
  static_assert(ROWS % RPP == 0 && ROWS <= 256, "whole passes; one modality byte per thread");
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  if (Ld.inplace || (ctl && ctl[1] != 0)) return;  // in-place layer, or a call that moves nothing
  const int Mv = eff[2 * l], M = Mv + eff[2 * l + 1];
  const int i0 = blockIdx.x * ROWS;
  if (i0 >= M) return;
  if (g == 0 && Ld.mod_out && threadIdx.x < ROWS && i0 + (int)threadIdx.x < M)
    Ld.mod_out[i0 + threadIdx.x] = i0 + (int)threadIdx.x < Mv ? 0 : 1;
  const int32_t* ig = idx + ((int64_t)l * dm.Hkv + g) * dm.max_tokens;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const T* v = reinterpret_cast<const T*>(Ld.v) + (int64_t)g * Ld.kv_hs;
  T* ko = reinterpret_cast<T*>(Ld.k_out) + (int64_t)g * Ld.out_hs;
  T* vo = reinterpret_cast<T*>(Ld.v_out) + (int64_t)g * Ld.out_hs;
  const int sub = threadIdx.x % CPR;
  constexpr int NP = ROWS / RPP;  // rows per lane, all loaded before the first store
  int src[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int i = i0 + threadIdx.x / CPR + p * RPP;
    src[p] = i < M ? ig[i] : -1;
  }
  uint4 kx[NP], vx[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    if ((unsigned)src[p] < (unsigned)Ld.n) {  // never read outside the working set
      kx[p] = gload16(k + (int64_t)src[p] * Ld.kv_rs + sub * (16 / sizeof(T)));
      vx[p] = gload16(v + (int64_t)src[p] * Ld.kv_rs + sub * (16 / sizeof(T)));
    }
  }
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int i = i0 + threadIdx.x / CPR + p * RPP;
    if ((unsigned)src[p] < (unsigned)Ld.n) {
      *reinterpret_cast<uint4*>(ko + (int64_t)i * Ld.out_rs + sub * (16 / sizeof(T))) = kx[p];
      *reinterpret_cast<uint4*>(vo + (int64_t)i * Ld.out_rs + sub * (16 / sizeof(T))) = vx[p];
    }
  }
}

// Inputs of layer-shared selection, one thread per working-set row: the
// layer's importance, a summed over the KV heads, and its redundancy, s
// summed over them and divided by their count (fp32, in head order).
__global__ __launch_bounds__(256) void layer_inputs(const LayerDesc* __restrict__ layers, Dims dm,
                                                    const float* __restrict__ a, const float* __restrict__ s,
                                                    float* __restrict__ la, float* __restrict__ ls) {
  const int l = blockIdx.y;
  const int j = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (j >= layers[l].n) return;
  float ta = 0.0f, ts = 0.0f;
  for (int h = 0; h < dm.Hkv; ++h) {
    const int64_t o = ((int64_t)l * dm.Hkv + h) * dm.max_tokens + j;
    ta += a[o];
    ts += s[o];
  }
  la[(int64_t)l * dm.max_tokens + j] = ta;
  ls[(int64_t)l * dm.max_tokens + j] = ts / (float)dm.Hkv;
}

// Kept rows' hidden states, for layers that give hidden_out (layer-shared
// selection: the index rows of all heads are equal, head 0's is read):
// hidden_out[i] = hidden[idx[l][0][i]], one wave per row, 16 bytes a lane.
template <typename T>
__global__ __launch_bounds__(256) void gather_hidden(const LayerDesc* __restrict__ layers, Dims dm,
                                                     const int32_t* __restrict__ idx, const int* __restrict__ eff,
                                                     const int* __restrict__ ctl) {
  const int l = blockIdx.y;
  const LayerDesc Ld = layers[l];
  if (!Ld.hidden_out || (ctl && ctl[1] != 0)) return;
  const int M = eff[2 * l] + eff[2 * l + 1];
  const int i = (int)blockIdx.x * 4 + wave_id(), lane = threadIdx.x & 63;
  if (i >= M) return;
  const int row = idx[(int64_t)l * dm.Hkv * dm.max_tokens + i];
  constexpr int EPP = 16 / (int)sizeof(T);
  const T* src = reinterpret_cast<const T*>(Ld.hidden) + (int64_t)row * Ld.hidden_rs;
  T* dst = reinterpret_cast<T*>(Ld.hidden_out) + (int64_t)i * Ld.hidden_out_rs;
  for (int c = lane; c < dm.dh / EPP; c += 64) *reinterpret_cast<uint4*>(dst + c * EPP) = gload16(src + c * EPP);
}

// ---------------------------------------------------------------------------
// Compaction in place (k_out, v_out are k, v).  Slot i of (layer, KV head)
// takes row p_i = idx[i].  Visual slots never take a row in front of them
// (p_i >= i: the i-th kept visual row has at least i rows before it), and
// neither do audio slots except a leading run of them, those whose row has
// fewer than M_v visual rows in front of it (M_v + j - p_j does not grow
// with j, so these are the first ones).  That run is copied out to the
// staging rows first (stage_moved_back); every other slot is then filled
// in one pass in which tile t (kGatherRows slots) writes its rows only after
// each earlier tile that reads one of those rows has loaded it (flags set after
// the loads).  The workgroups of one (layer, KV head) take its tiles as
// tickets from a counter of their own, in their order of starting, and the
// wait of a tile is only on tiles of the same (layer, KV head) with smaller
// tickets, whose loading phase waits for nothing: every wait ends.  One
// counter per (layer, KV head), each on a cache line of its own, keeps the
// ticket atomics from queueing on one address.
// ---------------------------------------------------------------------------
constexpr int kSpinLimit = 1 << 22;  // polls before a wait gives up (never reached when the order holds)
constexpr int kTicketStride = 32;    // ints between two ticket counters (one 128-byte line each)

// Rows of a tile, 16 bytes per lane: lane group `sub` of the row that
// thread t handles in pass p is t / CPR + p * RPP.
template <typename T, int D>
struct RowCopy {
  static constexpr int CPR = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  static constexpr int RPP = 256 / CPR;                // rows per pass
  static constexpr int NP = kGatherRows / RPP;         // passes
  static_assert(NP >= 1 && NP * RPP == kGatherRows, "whole passes of rows");
  static constexpr int EPC = 16 / (int)sizeof(T);
};

// Zero the read flags and ticket counters, and stage the slots that take a
// row in front of them.  Grid: (ceil(stage_rows / kGatherRows), H_kv, L);
// tile x stages the kGatherRows audio slots from M_v + kGatherRows x (the
// run that moves back is a prefix of the audio slots, so it lies in the
// first stage_rows of them unless it is too long) and zeroes every
// gridDim.x-th read flag.  The workgroup of tile 0 also checks the first
// slot past the staging rows; if that one moves back too, it counts the
// whole run (the shortfall) for the status word.
template <typename T, int D>
__global__ __launch_bounds__(256) void stage_moved_back(const LayerDesc* __restrict__ layers, Dims dm,
                                                        const int32_t* __restrict__ idx, const int* __restrict__ eff,
                                                        Workspace ws, int active) {
  using RC = RowCopy<T, D>;
  const int l = blockIdx.z, g = blockIdx.y;
  const int u = l * dm.Hkv + g;
  // (rotated by the unit, so that the few workgroups with rows to stage,
  // the first of each unit, spread over the XCDs)
  const int x = (int)((blockIdx.x + (unsigned)u) % gridDim.x);
  const int tiles = (int)((dm.max_tokens + kGatherRows - 1) / kGatherRows);
  for (int t = x * 256 + (int)threadIdx.x; t < active; t += (int)gridDim.x * 256) ws.read_flags[(int64_t)u * tiles + t] = 0;
  if (x == 0 && threadIdx.x == 0) ws.tickets[u * kTicketStride] = 0;
  const LayerDesc Ld = layers[l];
  if (!Ld.inplace) return;
  const int Mv = eff[2 * l], M = Mv + eff[2 * l + 1];
  const int32_t* ig = idx + (int64_t)u * dm.max_tokens;
  auto moves_back = [&](int i) {
    const int row = ig[i];
    return row >= 0 && row < i;
  };
  if (x == 0 && Mv + ws.stage_rows < M && moves_back(Mv + ws.stage_rows)) {  // (uniform)
    int run = ws.stage_rows;
    for (int i0 = Mv + ws.stage_rows; i0 < M; i0 += 256) {
      const int i = i0 + (int)threadIdx.x;
      run += __syncthreads_count(i < M && moves_back(i));
    }
    if (threadIdx.x == 0) atomicMax(&ws.ctl[1], run);
    return;
  }
  const int j0 = x * kGatherRows;
  const int jend = min(ws.stage_rows, M - Mv);
  if (j0 >= jend) return;
  const T* k = reinterpret_cast<const T*>(Ld.k) + (int64_t)g * Ld.kv_hs;
  const T* v = reinterpret_cast<const T*>(Ld.v) + (int64_t)g * Ld.kv_hs;
  const int64_t stage_len = (int64_t)dm.L * dm.Hkv * ws.stage_rows * D;
  T* sk = reinterpret_cast<T*>(ws.stage) + (int64_t)u * ws.stage_rows * D;
  T* sv = sk + stage_len;
  const int sub = threadIdx.x % RC::CPR;
#pragma unroll
  for (int p = 0; p < RC::NP; ++p) {
    const int j = j0 + (int)threadIdx.x / RC::CPR + p * RC::RPP;
    if (j >= jend) continue;
    const int i = Mv + j;
    const int row = ig[i];
    if (row >= i || row < 0) continue;  // moves to the front or stays
    const int64_t e = (int64_t)row * Ld.kv_rs + sub * RC::EPC;
    const uint4 kx = gload16(k + e), vx = gload16(v + e);
    *reinterpret_cast<uint4*>(sk + (int64_t)j * D + sub * RC::EPC) = kx;
    *reinterpret_cast<uint4*>(sv + (int64_t)j * D + sub * RC::EPC) = vx;
  }
}

// Grid: `active` workgroups per (layer, KV head), unit u = blockIdx.x % units;
// `tiles` is the row stride of the flag array.
template <typename T, int D>
__global__ __launch_bounds__(256) void gather_inplace(const LayerDesc* __restrict__ layers, Dims dm,
                                                      const int32_t* __restrict__ idx, const int* __restrict__ eff,
                                                      Workspace ws, int units, int tiles, int active) {
  using RC = RowCopy<T, D>;
  __shared__ int s_ticket;
  const int u = (int)(blockIdx.x % (unsigned)units);
  if (threadIdx.x == 0) s_ticket = atomicAdd(&ws.tickets[u * kTicketStride], 1);
  __syncthreads();
  const int tile = s_ticket;
  if (blockIdx.x == 0 && threadIdx.x == 0 && ws.ctl[1] > ws.ctl[2]) ws.ctl[2] = ws.ctl[1];  // largest shortfall
  if (tile >= active) return;
  const int l = u / dm.Hkv, g = u % dm.Hkv;
  const LayerDesc Ld = layers[l];
  if (!Ld.inplace || ws.ctl[1] != 0) return;
  const int Mv = eff[2 * l], M = Mv + eff[2 * l + 1];
  const int i0 = tile * kGatherRows;
  if (i0 >= M) return;  // no slot here, and no later tile waits for this one
  const int32_t* ig = idx + (int64_t)u * dm.max_tokens;
  T* k = static_cast<T*>(Ld.k_out) + (int64_t)g * Ld.kv_hs;  // in place: k_out is k
  T* v = static_cast<T*>(Ld.v_out) + (int64_t)g * Ld.kv_hs;
  const int64_t stage_len = (int64_t)dm.L * dm.Hkv * ws.stage_rows * D;
  const T* sk = reinterpret_cast<const T*>(ws.stage) + (int64_t)u * ws.stage_rows * D;
  const T* sv = sk + stage_len;
  const int sub = threadIdx.x % RC::CPR;

  // Loading phase: each slot's row, from the working set (a row at or
  // behind the slot) or from the staging rows.
  int slot[RC::NP];
  bool move[RC::NP];
  uint4 kx[RC::NP], vx[RC::NP];
#pragma unroll
  for (int p = 0; p < RC::NP; ++p) {
    const int i = i0 + (int)threadIdx.x / RC::CPR + p * RC::RPP;
    slot[p] = i;
    const int row = i < M ? ig[i] : i;
    move[p] = false;
    if (row > i && row < Ld.n) {
      const int64_t e = (int64_t)row * Ld.kv_rs + sub * RC::EPC;
      kx[p] = gload16(k + e);
      vx[p] = gload16(v + e);
      move[p] = true;
    } else if (row < i && row >= 0 && i >= Mv && i - Mv < ws.stage_rows) {
      const int64_t e = (int64_t)(i - Mv) * D + sub * RC::EPC;
      kx[p] = gload16(sk + e);
      vx[p] = gload16(sv + e);
      move[p] = true;
    }
  }
  dma_wait();        // this wave's loads have returned
  __syncthreads();   // ... and every other wave's
  if (threadIdx.x == 0)
    __hip_atomic_store(&ws.read_flags[(int64_t)u * tiles + tile], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // Each row this tile overwrites must have been loaded by the slot that
  // takes it: by this tile (the barrier above), by a staging copy (a later
  // slot), or by an earlier tile, whose flag is awaited here.
  if (threadIdx.x < kGatherRows) {
    const int i = i0 + (int)threadIdx.x;
    int wait_tile = -1;
    if (i < M && ig[i] != i) {
      const int reader = ws.slot_of[(int64_t)u * dm.max_tokens + i];
      if (reader >= 0 && reader < i0) wait_tile = reader / kGatherRows;
    }
    if (wait_tile >= 0) {
      const int* f = &ws.read_flags[(int64_t)u * tiles + wait_tile];
      int polls = 0;
      while (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
        __builtin_amdgcn_s_sleep(2);
        if (++polls == kSpinLimit) {
          atomicAdd(&ws.ctl[3], 1);
          break;
        }
      }
    }
  }
  __syncthreads();

  // Writing phase.
#pragma unroll
  for (int p = 0; p < RC::NP; ++p) {
    if (!move[p]) continue;
    const int64_t e = (int64_t)slot[p] * Ld.kv_rs + sub * RC::EPC;
    *reinterpret_cast<uint4*>(k + e) = kx[p];
    *reinterpret_cast<uint4*>(v + e) = vx[p];
  }
  if (g == 0 && Ld.mod_out && threadIdx.x < kGatherRows && i0 + (int)threadIdx.x < M)
    Ld.mod_out[i0 + threadIdx.x] = i0 + (int)threadIdx.x < Mv ? 0 : 1;
}

// Eq. (3): the chunk's K, V rows and modality behind each layer's retained
// rows; kAppendRows rows of one (layer, KV head) per workgroup (32 rows ran
// 6% faster than 64 on a 28-layer chunk, 128 rows 6% slower).
constexpr int kAppendRows = 32;
template <typename T, int D>
__global__ __launch_bounds__(256) void append_chunk(const LayerDesc* __restrict__ layers, Dims dm) {
  using RC = RowCopy<T, D>;
  constexpr int NP = kAppendRows / RC::RPP;  // passes
  static_assert(NP >= 1 && NP * RC::RPP == kAppendRows, "whole passes of rows");
  const int l = blockIdx.z, g = blockIdx.y;
  const LayerDesc Ld = layers[l];
  const int i0 = blockIdx.x * kAppendRows;
  if (i0 >= Ld.n_chunk) return;
  const T* ck = reinterpret_cast<const T*>(Ld.ck) + (int64_t)g * Ld.c_hs;
  const T* cv = reinterpret_cast<const T*>(Ld.cv) + (int64_t)g * Ld.c_hs;
  T* k = const_cast<T*>(reinterpret_cast<const T*>(Ld.k)) + (int64_t)g * Ld.kv_hs;
  T* v = const_cast<T*>(reinterpret_cast<const T*>(Ld.v)) + (int64_t)g * Ld.kv_hs;
  const int sub = threadIdx.x % RC::CPR;
  uint4 kx[NP], vx[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int i = i0 + (int)threadIdx.x / RC::CPR + p * RC::RPP;
    if (i < Ld.n_chunk) {
      const int64_t e = (int64_t)i * Ld.c_rs + sub * RC::EPC;
      kx[p] = gload16(ck + e);
      vx[p] = gload16(cv + e);
    }
  }
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int i = i0 + (int)threadIdx.x / RC::CPR + p * RC::RPP;
    if (i < Ld.n_chunk) {
      const int64_t e = (int64_t)(Ld.n_cache + i) * Ld.kv_rs + sub * RC::EPC;
      *reinterpret_cast<uint4*>(k + e) = kx[p];
      *reinterpret_cast<uint4*>(v + e) = vx[p];
    }
  }
  if (g == 0 && threadIdx.x < kAppendRows && i0 + (int)threadIdx.x < Ld.n_chunk) {
    uint8_t* mod = const_cast<uint8_t*>(Ld.mod);
    mod[Ld.n_cache + i0 + threadIdx.x] = gload<uint8_t>(Ld.cmod + i0 + threadIdx.x) ? 1 : 0;
  }
}

// inplace: 0 no layer in place, 1 some, 2 all.  max_n: the largest N of
// the call's layers (no layer keeps more rows).
template <typename T, int D>
void launch_gather(const Dims& dm, const LayerDesc* desc, const Workspace& ws, const int32_t* idx, int inplace,
                   int max_n, hipStream_t st) {
  const int tiles = (int)((dm.max_tokens + kGatherRows - 1) / kGatherRows);
  const int active = (max_n + kGatherRows - 1) / kGatherRows;
  const int* ctl = ws.stage_rows > 0 ? ws.ctl : nullptr;
  if (inplace < 2) {
    const dim3 grid((unsigned)((max_n + kCompactRows - 1) / kCompactRows), dm.Hkv, dm.L);
    OMNIMEM_LAUNCH(ws, K_GATHER, st, gather_compact<T, D><<<grid, 256, 0, st>>>(desc, dm, idx, ws.eff, ctl));
  }
  if (inplace > 0) {
    const int units = dm.L * dm.Hkv;
    const dim3 gstage((unsigned)max(1, (ws.stage_rows + kGatherRows - 1) / kGatherRows), dm.Hkv, dm.L);
    OMNIMEM_LAUNCH(ws, K_STAGE, st, stage_moved_back<T, D><<<gstage, 256, 0, st>>>(desc, dm, idx, ws.eff, ws, active));
    OMNIMEM_LAUNCH(ws, K_GATHER_IP, st,
                   gather_inplace<T, D><<<(unsigned)(units * active), 256, 0, st>>>(desc, dm, idx, ws.eff, ws,
                                                                                     units, tiles, active));
  }
}

template <bool SHARED>
void launch_topk(const Dims& dm, float lambda, int max_n, int path, const LayerDesc* desc, const Workspace& ws,
                 const float* a, const float* s, const int32_t* budgets, int32_t* ix, int* slot_of, int* ctl,
                 hipStream_t st) {
  const unsigned heads = SHARED ? 1u : (unsigned)dm.Hkv;
  if (path == OMNIMEM_TOPK_REGISTERS) {
    static_assert(kRegRows == kTopkRegRows, "the register path's rows");
    OMNIMEM_LAUNCH(ws, K_TOPK_REG, st,
                   psi_topk_reg<SHARED><<<dim3(2, heads, dm.L), kSelThreads, 0, st>>>(desc, dm, lambda, a, s, budgets,
                                                                                      ix, ws.eff, slot_of, ctl));
    return;
  }
  if (path != OMNIMEM_TOPK_SPLIT) {
    OMNIMEM_LAUNCH(ws, K_TOPK, st,
                   psi_topk<SHARED><<<dim3(2, heads, dm.L), kSelThreads, 0, st>>>(desc, dm, lambda, a, s, budgets,
                                                                                  ws.keys, ix, ws.eff, slot_of, ctl));
    return;
  }
  const unsigned hx = (unsigned)((max_n + kHistRows - 1) / kHistRows);
  const unsigned sx = (unsigned)((max_n + kTopkSlice - 1) / kTopkSlice);
  OMNIMEM_LAUNCH(ws, K_TOPK_HIST, st,
                 topk_hist<SHARED><<<dim3(hx, heads, dm.L), kTkThreads, 0, st>>>(desc, dm, lambda, a, s, ws.keys,
                                                                                ws.tk_hist, ws.tk_ccount, ctl));
  OMNIMEM_LAUNCH(ws, K_TOPK_BIN, st,
                 topk_bin<SHARED><<<dim3(sx, heads, dm.L), kTkThreads, 0, st>>>(desc, dm, ws.keys, ws.tk_hist, budgets,
                                                                               ws.tk_seg, ws.tk_slice, ws.tk_cand,
                                                                               ws.tk_ccount, ws.eff));
  OMNIMEM_LAUNCH(ws, K_TOPK_EMIT, st,
                 topk_emit<SHARED><<<dim3(sx, heads, dm.L), kTkThreads, 0, st>>>(desc, dm, ws.keys, ws.tk_hist,
                                                                                ws.tk_seg, ws.tk_slice, ws.tk_cand,
                                                                                ix, slot_of));
}

}  // namespace

hipError_t launch_select_compact(const Dims& dm, int dtype, float lambda, int shared, bool hidden, int inplace,
                                 int max_n, int topk_path, const LayerDesc* desc, const Workspace& ws,
                                 const float* a, const float* s, const int32_t* budgets, int32_t* idx,
                                 hipStream_t st) {
  int32_t* ix = idx ? idx : ws.idx;
  int* slot_of = inplace ? ws.slot_of : nullptr;
  int* ctl = ws.stage_rows > 0 ? ws.ctl : nullptr;
  if (shared) {
    float* la = ws.layer_as;
    float* ls = ws.layer_as + (size_t)dm.L * dm.max_tokens;
    const dim3 gtok((unsigned)((dm.max_tokens + 255) / 256), dm.L);
    OMNIMEM_LAUNCH(ws, K_LAYER_IN, st, layer_inputs<<<gtok, 256, 0, st>>>(desc, dm, a, s, la, ls));
    launch_topk<true>(dm, lambda, max_n, topk_path, desc, ws, la, ls, budgets, ix, slot_of, ctl, st);
  } else {
    launch_topk<false>(dm, lambda, max_n, topk_path, desc, ws, a, s, budgets, ix, slot_of, ctl, st);
  }
  if (dtype == 0) {
    if (dm.d == 128) launch_gather<uint16_t, 128>(dm, desc, ws, ix, inplace, max_n, st);
    else launch_gather<uint16_t, 64>(dm, desc, ws, ix, inplace, max_n, st);
  } else {
    if (dm.d == 128) launch_gather<float, 128>(dm, desc, ws, ix, inplace, max_n, st);
    else launch_gather<float, 64>(dm, desc, ws, ix, inplace, max_n, st);
  }
  if (hidden) {
    const dim3 grid((unsigned)((dm.max_tokens + 3) / 4), dm.L);
    if (dtype == 0)
      OMNIMEM_LAUNCH(ws, K_GATHER_H, st, gather_hidden<uint16_t><<<grid, 256, 0, st>>>(desc, dm, ix, ws.eff, ctl));
    else
      OMNIMEM_LAUNCH(ws, K_GATHER_H, st, gather_hidden<float><<<grid, 256, 0, st>>>(desc, dm, ix, ws.eff, ctl));
  }
  return hipGetLastError();
}

hipError_t launch_append(const Dims& dm, int dtype, const LayerDesc* desc, const Workspace& ws, int64_t max_rows,
                         hipStream_t st) {
  static_assert(kAppendRows <= 256, "one modality byte per thread");
  const dim3 grid((unsigned)((max_rows + kAppendRows - 1) / kAppendRows), dm.Hkv, dm.L);
  if (dtype == 0) {
    if (dm.d == 128) OMNIMEM_LAUNCH(ws, K_APPEND, st, append_chunk<uint16_t, 128><<<grid, 256, 0, st>>>(desc, dm));
    else OMNIMEM_LAUNCH(ws, K_APPEND, st, append_chunk<uint16_t, 64><<<grid, 256, 0, st>>>(desc, dm));
  } else {
    if (dm.d == 128) OMNIMEM_LAUNCH(ws, K_APPEND, st, append_chunk<float, 128><<<grid, 256, 0, st>>>(desc, dm));
    else OMNIMEM_LAUNCH(ws, K_APPEND, st, append_chunk<float, 64><<<grid, 256, 0, st>>>(desc, dm));
  }
  return hipGetLastError();
}

}  // namespace omnimem
