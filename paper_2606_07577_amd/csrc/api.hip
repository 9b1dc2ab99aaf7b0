// Host side of the C ABI in include/omnimem.h: argument validation,
// workspace ownership, descriptor upload and the launch sequence of each
// stage.  No device memory is allocated after omnimem_create.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/omnimem.h"
#include "common.h"

using namespace omnimem;

namespace {

constexpr int kSlots = 16;        // descriptor ring depth
constexpr int64_t kTopkAutoSplitRows = 16384;  // longest working set AUTO ranks in one workgroup
constexpr int kProfEvents = 2 * 16384;
constexpr int kMaxLayers = 1024;  // bound of the allocation kernel's tables

std::string g_create_error;

}  // namespace

// Scratch of omnimem_allocate_noalloc (see there).
constexpr size_t kScratchBytes = (size_t)4 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace omnimem {
// Launch timing: an event pool and the (kernel, begin event) of each launch.
struct Profiler {
  std::vector<hipEvent_t> pool;
  int used = 0;
  std::vector<int> kernel;   // per recorded launch
  std::vector<int> first;    // index of its begin event; end event is first + 1
  bool open = false;
};

void prof_mark(Profiler* p, int kid, hipStream_t st, bool begin) {
  if (begin) {
    if (p->used + 2 > (int)p->pool.size()) return;
    if (hipEventRecord(p->pool[p->used], st) != hipSuccess) return;
    p->kernel.push_back(kid);
    p->first.push_back(p->used);
    p->used += 2;
    p->open = true;
  } else if (p->open) {
    (void)hipEventRecord(p->pool[p->first.back() + 1], st);
    p->open = false;
  }
}
}  // namespace omnimem

static const char* kKernelNames[K_COUNT] = {
    "lse_pass", "lse_merge", "colsum_pass", "head_sum", "modality_lists", "lists_norms", "gram_pass", "gram_finish", "adjacent_cos", "avba_partials", "avba_allocate", "psi_topk", "gather_compact",
    "gather_hidden", "adjacent_cos_hidden", "hidden_norms", "gram_wide", "hidden_finish", "layer_inputs",
    "stage_moved_back", "gather_inplace", "append_chunk", "gram_sym", "topk_hist", "topk_bin", "topk_emit", "psi_topk_reg"};

struct omnimem_ctx {
  omnimem_config cfg;
  Dims dm;
  int device = 0;
  Workspace ws{};
  LayerDesc* pinned = nullptr;          // host ring [kSlots][L]
  hipEvent_t ev[kSlots] = {};
  bool ev_used[kSlots] = {};
  int next_slot = 0;
  int last_slot = -1;                   // slot holding the last uploaded table
  std::vector<LayerDesc> last_table;
  PassPlan lse_plan{0, 0}, cs_plan{0, 0};  // score-pass plans of the last table
  int max_workgroups = 512;               // persistent score-pass grid: 2 per compute unit
  int calib_steps = 0;                    // steps in the calibration sums since the last reset
  int topk_path = OMNIMEM_TOPK_AUTO;
  std::string err;
  std::vector<void*> allocations;
  Profiler prof;
};

namespace {

omnimem_status fail(omnimem_ctx* ctx, omnimem_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx) ctx->err = buf; else g_create_error = buf;
  return st;
}

omnimem_status hip_fail(omnimem_ctx* ctx, hipError_t e, const char* where) {
  return fail(ctx, OMNIMEM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

size_t elt_size(const omnimem_config& c) { return c.dtype == OMNIMEM_BF16 ? 2 : 4; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Byte range [lo, hi) covered by a [heads][rows][d] strided tensor.
void extent(const void* base, int64_t heads, int64_t rows, int64_t hs, int64_t rs, int64_t d, size_t esz,
            uintptr_t* lo, uintptr_t* hi) {
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  const int64_t last = (heads - 1) * hs + (rows - 1) * rs + d;
  *lo = b;
  *hi = b + (uintptr_t)(last * (int64_t)esz);
}

bool overlaps(uintptr_t a0, uintptr_t a1, uintptr_t b0, uintptr_t b1) { return a0 < b1 && b0 < a1; }

enum Need { NEED_Q = 1, NEED_K = 2, NEED_V = 4, NEED_OUT = 8 };

// Compaction in place: the outputs are the working set itself.
bool in_place(const omnimem_layer& L) {
  return L.k_out == L.k && L.v_out == L.v && L.out_head_stride == L.kv_head_stride &&
         L.out_row_stride == L.kv_row_stride;
}

omnimem_status validate(omnimem_ctx* ctx, const omnimem_layer* layers, int need) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  if (!layers) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null layer array");
  const omnimem_config& c = ctx->cfg;
  const int64_t d = c.head_dim;
  const size_t esz = elt_size(c);
  for (int l = 0; l < c.n_layers; ++l) {
    const omnimem_layer& L = layers[l];
    const int64_t n = L.n_cache + L.n_chunk;
    if (L.n_cache < 0 || L.n_chunk < 0 || n < 1)
      return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: need n_cache >= 0, n_chunk >= 0, N >= 1", l);
    if (n > c.max_tokens || L.n_chunk > c.max_chunk)
      return fail(ctx, OMNIMEM_ERR_CAPACITY, "layer %d: N=%lld or n_chunk=%lld beyond the context's capacity", l,
                  (long long)n, (long long)L.n_chunk);
    if (!L.modality) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: null modality", l);
    if (!std::isfinite(L.sm_scale)) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: sm_scale not finite", l);
    if ((need & NEED_Q)) {
      if (!L.q) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: null q", l);
      if (!aligned16(L.q) || L.q_row_stride < d || L.q_head_stride < 0 || (L.q_row_stride * esz) % 16 ||
          (L.q_head_stride * esz) % 16)
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: q must be 16-byte aligned with row stride >= d and "
                    "strides of whole 16-byte units", l);
      if (L.lse && (reinterpret_cast<uintptr_t>(L.lse) & 3u))
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: lse not 4-byte aligned", l);
    }
    const bool need_k = need & NEED_K, need_v = need & NEED_V;
    if ((need_k && !L.k) || (need_v && !L.v)) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: null k or v", l);
    if (need_k || need_v) {
      if ((L.k && !aligned16(L.k)) || (L.v && !aligned16(L.v)) || L.kv_row_stride < d || L.kv_head_stride < 0 ||
          (L.kv_row_stride * esz) % 16 || (L.kv_head_stride * esz) % 16)
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: k/v must be 16-byte aligned with row stride >= d and "
                    "strides of whole 16-byte units", l);
      // bf16 rows are addressed by 32-bit byte offsets from a head's base
      const int64_t rs_b = L.kv_row_stride * (int64_t)esz;
      if (c.dtype == OMNIMEM_BF16 && (rs_b >= (int64_t{1} << 24) || rs_b * c.max_tokens >= (int64_t{1} << 31)))
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: bf16 k/v need a row stride below 16 MiB and row "
                    "stride x max_tokens below 2 GiB", l);
    }
    if (need & NEED_OUT) {
      if (!L.k_out || !L.v_out) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: null k_out or v_out", l);
      if (L.out_rows < 0) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: out_rows < 0", l);
      const int64_t H = c.n_kv_heads;
      const int64_t cap = L.out_rows ? L.out_rows : n;
      uintptr_t k0, k1, v0, v1, o0, o1, p0, p1;
      extent(L.k, H, n, L.kv_head_stride, L.kv_row_stride, d, esz, &k0, &k1);
      extent(L.v, H, n, L.kv_head_stride, L.kv_row_stride, d, esz, &v0, &v1);
      if (in_place(L)) {
        if (c.inplace_stage_rows <= 0)
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: k_out/v_out are k/v (in place), but the context "
                      "reserves no staging rows (inplace_stage_rows = 0)", l);
        if (overlaps(k0, k1, v0, v1))
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: in place, k and v must not overlap", l);
        o0 = k0; o1 = k1; p0 = v0; p1 = v1;
      } else {
        if (!aligned16(L.k_out) || !aligned16(L.v_out) || (L.out_row_stride * esz) % 16 ||
            (L.out_head_stride * esz) % 16)
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: outputs must be 16-byte aligned, strides of whole "
                      "16-byte units", l);
        const bool head_major = L.out_row_stride >= d && (H == 1 || L.out_head_stride >= cap * L.out_row_stride);
        const bool row_major = L.out_head_stride >= d && L.out_row_stride >= H * L.out_head_stride;
        if (!head_major && !row_major)
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: k_out/v_out must hold H_kv x out_rows rows of d "
                      "without overlap", l);
        extent(L.k_out, H, cap, L.out_head_stride, L.out_row_stride, d, esz, &o0, &o1);
        extent(L.v_out, H, cap, L.out_head_stride, L.out_row_stride, d, esz, &p0, &p1);
        if (overlaps(o0, o1, k0, k1) || overlaps(o0, o1, v0, v1) || overlaps(p0, p1, k0, k1) ||
            overlaps(p0, p1, v0, v1) || overlaps(o0, o1, p0, p1))
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: k_out/v_out overlap k, v or each other without "
                      "being k and v themselves", l);
      }
      if (L.modality_out) {
        const uintptr_t m0 = reinterpret_cast<uintptr_t>(L.modality_out), m1 = m0 + (uintptr_t)cap;
        const uintptr_t i0 = reinterpret_cast<uintptr_t>(L.modality), i1 = i0 + (uintptr_t)n;
        if ((m0 != i0 && overlaps(m0, m1, i0, i1)) || overlaps(m0, m1, o0, o1) || overlaps(m0, m1, p0, p1))
          return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: modality_out overlaps the outputs, or the input "
                      "modality without being it", l);
      }
    }
  }
  return OMNIMEM_OK;
}

// Hidden-state rows of each layer (the redundancy source of Eq. 7 as
// printed) and, for select_compact, their optional output rows.
omnimem_status validate_hidden(omnimem_ctx* ctx, const omnimem_layer* layers, bool outputs) {
  const omnimem_config& c = ctx->cfg;
  const int64_t dh = c.hidden_dim;
  const size_t esz = elt_size(c);
  for (int l = 0; l < c.n_layers; ++l) {
    const omnimem_layer& L = layers[l];
    const int64_t n = L.n_cache + L.n_chunk;
    if (!outputs || L.hidden_out) {
      if (!L.hidden || !aligned16(L.hidden) || L.hidden_row_stride < dh || (L.hidden_row_stride * esz) % 16)
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: hidden states must be given, 16-byte aligned, with "
                    "row stride >= hidden_dim in whole 16-byte units", l);
    }
    if (outputs && L.hidden_out) {
      if (!c.shared_selection)
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: kept hidden states need shared_selection (one index "
                    "set per layer)", l);
      if (!aligned16(L.hidden_out) || L.hidden_out_row_stride < dh || (L.hidden_out_row_stride * esz) % 16)
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: hidden_out must be 16-byte aligned with row stride "
                    ">= hidden_dim in whole 16-byte units", l);
      uintptr_t h0, h1, o0, o1;
      extent(L.hidden, 1, n, 0, L.hidden_row_stride, dh, esz, &h0, &h1);
      extent(L.hidden_out, 1, n, 0, L.hidden_out_row_stride, dh, esz, &o0, &o1);
      if (overlaps(o0, o1, h0, h1))
        return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: hidden_out overlaps hidden", l);
    }
  }
  return OMNIMEM_OK;
}

// New chunk rows of each layer (omnimem_append).
omnimem_status validate_append(omnimem_ctx* ctx, const omnimem_layer* layers, const omnimem_chunk* chunks) {
  if (!chunks) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null chunk array");
  const omnimem_config& c = ctx->cfg;
  const int64_t d = c.head_dim, H = c.n_kv_heads;
  const size_t esz = elt_size(c);
  for (int l = 0; l < c.n_layers; ++l) {
    const omnimem_layer& L = layers[l];
    const omnimem_chunk& C = chunks[l];
    if (C.n_rows != L.n_chunk)
      return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: chunk has %lld rows, the descriptor's n_chunk is %lld", l,
                  (long long)C.n_rows, (long long)L.n_chunk);
    if (L.n_chunk == 0) continue;
    if (!C.k || !C.v || !C.modality)
      return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: null chunk k, v or modality", l);
    if (!aligned16(C.k) || !aligned16(C.v) || C.row_stride < d || C.head_stride < 0 || (C.row_stride * esz) % 16 ||
        (C.head_stride * esz) % 16)
      return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: chunk k/v must be 16-byte aligned with row stride >= d "
                  "and strides of whole 16-byte units", l);
    const char* kd = static_cast<const char*>(L.k) + L.n_cache * L.kv_row_stride * (int64_t)esz;
    const char* vd = static_cast<const char*>(L.v) + L.n_cache * L.kv_row_stride * (int64_t)esz;
    uintptr_t a0, a1, b0, b1, x0, x1, y0, y1;
    extent(kd, H, L.n_chunk, L.kv_head_stride, L.kv_row_stride, d, esz, &a0, &a1);
    extent(vd, H, L.n_chunk, L.kv_head_stride, L.kv_row_stride, d, esz, &b0, &b1);
    extent(C.k, H, L.n_chunk, C.head_stride, C.row_stride, d, esz, &x0, &x1);
    extent(C.v, H, L.n_chunk, C.head_stride, C.row_stride, d, esz, &y0, &y1);
    const uintptr_t m0 = reinterpret_cast<uintptr_t>(L.modality) + (uintptr_t)L.n_cache, m1 = m0 + L.n_chunk;
    const uintptr_t c0 = reinterpret_cast<uintptr_t>(C.modality), c1 = c0 + L.n_chunk;
    if (overlaps(a0, a1, b0, b1) || overlaps(a0, a1, x0, x1) || overlaps(a0, a1, y0, y1) ||
        overlaps(b0, b1, x0, x1) || overlaps(b0, b1, y0, y1) || overlaps(m0, m1, c0, c1))
      return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "layer %d: the chunk rows overlap the rows they are copied to, or "
                  "the destination k and v rows overlap", l);
  }
  return OMNIMEM_OK;
}

// Device descriptor of one layer (the score-pass plan fields are filled by
// plan_score).
void describe(const omnimem_config& cfg, const omnimem_layer& s, const omnimem_chunk* chunk, LayerDesc* out) {
  LayerDesc& x = *out;
  std::memset(&x, 0, sizeof x);
  x.q = s.q; x.k = s.k; x.v = s.v; x.mod = s.modality; x.lse_in = s.lse;
  x.k_out = s.k_out; x.v_out = s.v_out;
  x.q_hs = s.q_head_stride; x.q_rs = s.q_row_stride;
  x.kv_hs = s.kv_head_stride; x.kv_rs = s.kv_row_stride;
  x.out_hs = s.out_head_stride; x.out_rs = s.out_row_stride;
  if (cfg.sim_source == OMNIMEM_SRC_HIDDEN) {
    x.hidden = s.hidden; x.hidden_out = s.hidden_out;
    x.hidden_rs = s.hidden_row_stride; x.hidden_out_rs = s.hidden_out_row_stride;
  }
  x.n_cache = (int32_t)s.n_cache; x.n_chunk = (int32_t)s.n_chunk; x.n = (int32_t)(s.n_cache + s.n_chunk);
  x.mod_out = s.modality_out;
  x.out_cap = (int32_t)std::min<int64_t>(s.out_rows > 0 ? s.out_rows : x.n, x.n);
  x.inplace = (s.k_out && in_place(s)) ? 1 : 0;
  if (chunk) {
    x.ck = chunk->k; x.cv = chunk->v; x.cmod = chunk->modality;
    x.c_hs = chunk->head_stride; x.c_rs = chunk->row_stride;
  }
  const double log2e = 1.4426950408889634;
  const double scale = s.sm_scale != 0.0f ? (double)s.sm_scale : 1.0 / std::sqrt((double)cfg.head_dim);
  x.scale_log2 = (float)(scale * log2e);
}

// Copy the descriptor table to the device unless it equals the last one.
omnimem_status upload(omnimem_ctx* ctx, const omnimem_layer* layers, hipStream_t st, const LayerDesc** dev,
                      const omnimem_chunk* chunks = nullptr) {
  const int L = ctx->cfg.n_layers;
  std::vector<LayerDesc> t(L);
  for (int l = 0; l < L; ++l) {
    describe(ctx->cfg, layers[l], chunks ? &chunks[l] : nullptr, &t[l]);
  }
  plan_score(ctx->dm, t.data(), ctx->max_workgroups, &ctx->lse_plan, &ctx->cs_plan);
  if (ctx->last_slot >= 0 && ctx->last_table.size() == t.size() &&
      std::memcmp(ctx->last_table.data(), t.data(), sizeof(LayerDesc) * L) == 0) {
    *dev = ctx->ws.desc + (size_t)ctx->last_slot * L;
    return OMNIMEM_OK;
  }
  const int slot = ctx->next_slot;
  if (ctx->ev_used[slot]) {
    hipError_t e = hipEventSynchronize(ctx->ev[slot]);
    if (e != hipSuccess) return hip_fail(ctx, e, "descriptor ring wait");
  }
  LayerDesc* host = ctx->pinned + (size_t)slot * L;
  std::memcpy(host, t.data(), sizeof(LayerDesc) * L);
  LayerDesc* d = ctx->ws.desc + (size_t)slot * L;
  hipError_t e = hipMemcpyAsync(d, host, sizeof(LayerDesc) * L, hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(ctx, e, "descriptor upload");
  ctx->last_slot = slot;
  ctx->last_table = t;
  ctx->next_slot = (slot + 1) % kSlots;
  *dev = d;
  return OMNIMEM_OK;
}

// Mark the slot in use by this call's work.
omnimem_status finish(omnimem_ctx* ctx, hipError_t launch_err, hipStream_t st, const char* what) {
  if (launch_err != hipSuccess) return hip_fail(ctx, launch_err, what);
  const int slot = ctx->last_slot;
  hipError_t e = hipEventRecord(ctx->ev[slot], st);
  if (e != hipSuccess) return hip_fail(ctx, e, "event record");
  ctx->ev_used[slot] = true;
  ctx->err.clear();
  return OMNIMEM_OK;
}

omnimem_status set_device(omnimem_ctx* ctx) {
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
  e = hipGetLastError();  // an earlier asynchronous fault surfaces here
  if (e != hipSuccess) return hip_fail(ctx, e, "earlier device error");
  return OMNIMEM_OK;
}

// Sizes and options of a configuration, checked without touching the device.
omnimem_status check_config(const omnimem_config& c) {
  if (c.n_layers < 1 || c.n_layers > kMaxLayers || c.n_q_heads < 1 || c.n_kv_heads < 1 ||
      c.n_q_heads % c.n_kv_heads != 0 || c.max_tokens < 1 || c.max_chunk < 0 || c.max_chunk > c.max_tokens ||
      c.max_tokens > (int64_t)1 << 30)
    return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "bad sizes: need 1 <= n_layers <= %d, H_kv | H_q, "
                "0 <= max_chunk <= max_tokens <= 2^30", kMaxLayers);
  if ((int64_t)c.n_layers * c.n_kv_heads > 256)
    return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "n_layers * n_kv_heads = %d: at most 256 supported",
                c.n_layers * c.n_kv_heads);
  if (c.head_dim != 64 && c.head_dim != 128)
    return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "head_dim %d: supported 64 and 128", c.head_dim);
  if (c.dtype != OMNIMEM_BF16 && c.dtype != OMNIMEM_F32)
    return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "dtype %d", c.dtype);
  if (c.sim != OMNIMEM_SIM_MAX && c.sim != OMNIMEM_SIM_ADJ)
    return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "sim %d", c.sim);
  if (c.sim_source < OMNIMEM_SRC_VALUES || c.sim_source > OMNIMEM_SRC_HIDDEN)
    return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "sim_source %d", c.sim_source);
  if (c.sim_source == OMNIMEM_SRC_HIDDEN) {
    const int64_t esz = c.dtype == OMNIMEM_BF16 ? 2 : 4;
    if (c.hidden_dim < 1 || c.hidden_dim > 65536 || (c.hidden_dim * esz) % 16)
      return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "hidden_dim %d: need 1..65536 and rows of whole 16-byte units",
                  c.hidden_dim);
    if (c.sim == OMNIMEM_SIM_MAX && c.hidden_dim % 64)
      return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "hidden_dim %d: the all-pairs maximum on hidden states takes "
                  "multiples of 64", c.hidden_dim);
  }
  if (c.inplace_stage_rows < 0 || c.inplace_stage_rows > c.max_tokens)
    return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "inplace_stage_rows %d: need 0 .. max_tokens", c.inplace_stage_rows);
  if (!std::isfinite(c.lambda) || c.lambda < 0.0f || !(c.ratio_r > 0.0f) || !(c.temperature > 0.0f) ||
      !(c.b_min_frac >= 0.0f) || !(c.b_max_frac >= c.b_min_frac) || !std::isfinite(c.b_max_frac))
    return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "need lambda >= 0, r > 0, T > 0, 0 <= b_min_frac <= b_max_frac");
  return OMNIMEM_OK;
}

Dims make_dims(const omnimem_config& c) {
  Dims dm;
  dm.L = c.n_layers; dm.Hq = c.n_q_heads; dm.Hkv = c.n_kv_heads; dm.G = c.n_q_heads / c.n_kv_heads;
  dm.d = c.head_dim; dm.max_tokens = c.max_tokens; dm.max_chunk = std::max<int64_t>(c.max_chunk, 1);
  dm.causal = c.causal ? 1 : 0;
  dm.qb = (int)((dm.max_chunk + kScoreBlock - 1) / kScoreBlock);
  dm.kb = (int)((dm.max_tokens + kScoreBlock - 1) / kScoreBlock);
  dm.dh = c.sim_source == OMNIMEM_SRC_HIDDEN ? c.hidden_dim : 0;
  return dm;
}

// Arguments of the allocation stage (Eqs. 9-14), including the host-side
// feasibility of the per-layer minimum budgets.
omnimem_status check_allocate(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a, const float* s,
                              int64_t total_budget, const int32_t* budgets) {
  omnimem_status st = validate(ctx, layers, 0);
  if (st != OMNIMEM_OK) return st;
  if (!a || !s || !budgets) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null a, s or budgets");
  const omnimem_config& c = ctx->cfg;
  if (total_budget < 0 || total_budget > ((int64_t)1 << 40))
    return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "total budget %lld out of range", (long long)total_budget);
  const int64_t lo_base = (int64_t)std::ceil(((double)c.b_min_frac * (double)total_budget) / c.n_layers);
  int64_t sum_lo = 0;
  for (int l = 0; l < c.n_layers; ++l) sum_lo += std::min<int64_t>(lo_base, layers[l].n_cache + layers[l].n_chunk);
  if (sum_lo > total_budget)
    return fail(ctx, OMNIMEM_ERR_INFEASIBLE, "per-layer minimum budgets sum to %lld > total %lld",
                (long long)sum_lo, (long long)total_budget);
  return OMNIMEM_OK;
}

// ---------------------------------------------------------------------------
// The allocation stage without a context and without any device allocation
// (omnimem_allocate_noalloc).  Its scratch -- the layer table and the fp64
// partial sums of Eqs. 9-10 and 13 -- lives in `scratch`, a fixed device
// array of kScratchBytes that every GPU the library runs on holds until the
// process ends.  Host code never uses the array's name as an address: the
// first call on a device asks the runtime for the array's address on that
// device (hipGetSymbolAddress, with the device current) and keeps it.
// ---------------------------------------------------------------------------
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

omnimem_status scratch_address(int device, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (device < 0 || device >= kMaxDevices)
    return fail(nullptr, OMNIMEM_ERR_UNSUPPORTED, "device %d: at most %d devices", device, kMaxDevices);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(nullptr, OMNIMEM_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return OMNIMEM_OK;
}

// Layer descriptors passed by value and stored into the scratch table.
constexpr int kDescPerStore = 8;
struct DescBlock {
  LayerDesc d[kDescPerStore];
};
static_assert(sizeof(DescBlock) <= 3072, "kernel argument block too large");

__global__ void store_descs(LayerDesc* __restrict__ dst, DescBlock blk, int count) {
  if (threadIdx.x != 0) return;
#pragma unroll
  for (int i = 0; i < kDescPerStore; ++i)
    if (i < count) dst[i] = blk.d[i];
}

template <typename T>
hipError_t dalloc(omnimem_ctx* ctx, T** p, size_t count) {
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, std::max<size_t>(count * sizeof(T), 256));
  if (e == hipSuccess) ctx->allocations.push_back(q);
  *p = static_cast<T*>(q);
  return e;
}


}  // namespace

extern "C" {

void omnimem_config_default(omnimem_config* c) {
  if (!c) return;
  std::memset(c, 0, sizeof *c);
  c->dtype = OMNIMEM_BF16;
  c->lambda = 0.02f;
  c->ratio_r = 5.0f;
  c->temperature = 0.2f;
  c->b_min_frac = 0.5f;
  c->b_max_frac = 2.0f;
  c->causal = 1;
  c->sim = OMNIMEM_SIM_MAX;
  c->sim_source = OMNIMEM_SRC_VALUES;
  c->hidden_dim = 0;
}

omnimem_status omnimem_create(const omnimem_config* cfg, omnimem_ctx** out) {
  if (!cfg || !out) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  const omnimem_config& c = *cfg;
  omnimem_status cst = check_config(c);
  if (cst != OMNIMEM_OK) return cst;

  omnimem_ctx* ctx = new omnimem_ctx();
  ctx->cfg = c;
  hipError_t e = hipGetDevice(&ctx->device);
  if (e != hipSuccess) { delete ctx; return fail(nullptr, OMNIMEM_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e)); }
  Dims& dm = ctx->dm;
  dm = make_dims(c);
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, ctx->device) == hipSuccess && cus > 0)
    ctx->max_workgroups = 2 * cus;
  const size_t L = c.n_layers, Hq = c.n_q_heads, Hkv = c.n_kv_heads, T = c.max_tokens, Cm = dm.max_chunk;
  Workspace& ws = ctx->ws;
  ws.gram_grid = ctx->max_workgroups;
  ws.stage_rows = c.inplace_stage_rows;
  const size_t elt = c.dtype == OMNIMEM_BF16 ? 2 : 4;
  if ((e = dalloc(ctx, &ws.desc, (size_t)kSlots * L)) != hipSuccess ||
      (e = dalloc(ctx, &ws.lse_part, L * Hq * (size_t)dm.qb * kMaxSeg * kScoreBlock)) != hipSuccess ||
      (e = dalloc(ctx, &ws.lse2, L * Hq * Cm)) != hipSuccess ||
      (e = dalloc(ctx, &ws.part, L * Hq * (size_t)dm.kb * kMaxSeg * kScoreBlock)) != hipSuccess ||
      (e = dalloc(ctx, &ws.pos, L * 2 * (size_t)list_stride(T))) != hipSuccess ||
      (e = dalloc(ctx, &ws.rank, L * T)) != hipSuccess ||
      (e = dalloc(ctx, &ws.counts, L * 2)) != hipSuccess ||
      (e = dalloc(ctx, &ws.inv_norm, L * Hkv * T)) != hipSuccess ||
      (e = dalloc(ctx, &ws.best, L * Hkv * T)) != hipSuccess ||
      (c.dtype != OMNIMEM_BF16 &&  // fp32 rows are copied in segment order for the Gram pass
       (e = dalloc(ctx, reinterpret_cast<char**>(&ws.perm), L * Hkv * T * (size_t)c.head_dim * elt)) != hipSuccess) ||
      (e = dalloc(ctx, &ws.stat_part, L * Hkv * (size_t)allocate_part_chunks(dm) * 2 * 4)) != hipSuccess ||
      (e = dalloc(ctx, &ws.calib, L)) != hipSuccess ||
      (e = dalloc(ctx, &ws.eff, L * 2)) != hipSuccess ||
      (e = dalloc(ctx, &ws.idx, L * Hkv * T)) != hipSuccess ||
      (e = dalloc(ctx, &ws.keys, L * Hkv * (size_t)topk_stride(T))) != hipSuccess ||
      (e = dalloc(ctx, &ws.tk_hist, L * Hkv * 2 * (size_t)kTopkBins)) != hipSuccess ||
      (e = dalloc(ctx, &ws.tk_seg, L * Hkv * 2 * 8)) != hipSuccess ||
      (e = dalloc(ctx, &ws.tk_slice, L * Hkv * (size_t)kTopkMaxSlices * 2)) != hipSuccess ||
      (e = dalloc(ctx, &ws.tk_cand, L * Hkv * (size_t)topk_stride(T))) != hipSuccess ||
      (e = dalloc(ctx, &ws.tk_ccount, L * Hkv * 2)) != hipSuccess ||
      (c.shared_selection && (e = dalloc(ctx, &ws.layer_as, 2 * L * T)) != hipSuccess) ||
      (e = dalloc(ctx, &ws.ctl, 4)) != hipSuccess ||
      (c.inplace_stage_rows > 0 &&
       ((e = dalloc(ctx, reinterpret_cast<char**>(&ws.stage),
                    2 * L * Hkv * (size_t)c.inplace_stage_rows * (size_t)c.head_dim * elt)) != hipSuccess ||
        (e = dalloc(ctx, &ws.slot_of, L * Hkv * T)) != hipSuccess ||
        (e = dalloc(ctx, &ws.read_flags, L * Hkv * (size_t)((T + kGatherRows - 1) / kGatherRows))) != hipSuccess ||
        (e = dalloc(ctx, &ws.tickets, L * Hkv * 32)) != hipSuccess))) {
    omnimem_destroy(ctx);
    return fail(nullptr, OMNIMEM_ERR_HIP, "workspace allocation: %s", hipGetErrorString(e));
  }
  void* pinned = nullptr;
  if ((e = hipHostMalloc(&pinned, sizeof(LayerDesc) * kSlots * L, hipHostMallocDefault)) != hipSuccess) {
    omnimem_destroy(ctx);
    return fail(nullptr, OMNIMEM_ERR_HIP, "pinned descriptor ring: %s", hipGetErrorString(e));
  }
  ctx->pinned = static_cast<LayerDesc*>(pinned);
  if ((e = hipMemset(ws.ctl, 0, 4 * sizeof(int))) != hipSuccess ||
      (e = hipMemset(ws.tk_hist, 0, L * Hkv * 2 * (size_t)kTopkBins * sizeof(int))) != hipSuccess) {
    omnimem_destroy(ctx);
    return fail(nullptr, OMNIMEM_ERR_HIP, "control words: %s", hipGetErrorString(e));
  }
  for (int i = 0; i < kSlots; ++i) {
    if ((e = hipEventCreateWithFlags(&ctx->ev[i], hipEventDisableTiming)) != hipSuccess) {
      omnimem_destroy(ctx);
      return fail(nullptr, OMNIMEM_ERR_HIP, "event: %s", hipGetErrorString(e));
    }
  }
  *out = ctx;
  return OMNIMEM_OK;
}

omnimem_status omnimem_destroy(omnimem_ctx* ctx) {
  if (!ctx) return OMNIMEM_OK;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  for (void* p : ctx->allocations) (void)hipFree(p);
  if (ctx->pinned) (void)hipHostFree(ctx->pinned);
  for (int i = 0; i < kSlots; ++i)
    if (ctx->ev[i]) (void)hipEventDestroy(ctx->ev[i]);
  for (hipEvent_t e : ctx->prof.pool) (void)hipEventDestroy(e);
  delete ctx;
  return OMNIMEM_OK;
}

const char* omnimem_last_error(const omnimem_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

omnimem_status omnimem_score(omnimem_ctx* ctx, const omnimem_layer* layers, float* a, float* lse_out,
                             hipStream_t stream) {
  omnimem_status st = validate(ctx, layers, NEED_Q | NEED_K);
  if (st != OMNIMEM_OK) return st;
  if (!a) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null a");
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  return finish(ctx, launch_score(ctx->dm, ctx->cfg.dtype, dev, ctx->ws, ctx->lse_plan, ctx->cs_plan, lse_out, a,
                                  stream),
                stream, "omnimem_score launch");
}

omnimem_status omnimem_redundancy(omnimem_ctx* ctx, const omnimem_layer* layers, float* s, hipStream_t stream) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  const int src = ctx->cfg.sim_source;
  omnimem_status st = validate(ctx, layers, src == OMNIMEM_SRC_KEYS ? NEED_K : src == OMNIMEM_SRC_VALUES ? NEED_V : 0);
  if (st != OMNIMEM_OK) return st;
  if (!s) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null s");
  if (src == OMNIMEM_SRC_HIDDEN && (st = validate_hidden(ctx, layers, false)) != OMNIMEM_OK) return st;
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  return finish(ctx, launch_redundancy(ctx->dm, ctx->cfg.dtype, ctx->cfg.sim, ctx->cfg.sim_source, dev, ctx->ws,
                                       s, stream),
                stream, "omnimem_redundancy launch");
}

omnimem_status omnimem_allocate(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a, const float* s,
                                int64_t total_budget, int32_t* budgets, float* stats, hipStream_t stream) {
  omnimem_status st = check_allocate(ctx, layers, a, s, total_budget, budgets);
  if (st != OMNIMEM_OK) return st;
  const omnimem_config& c = ctx->cfg;
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  return finish(ctx, launch_allocate(ctx->dm, dev, ctx->ws, a, s, total_budget, c.ratio_r, c.temperature,
                                     c.b_min_frac, c.b_max_frac, budgets, stats, stream),
                stream, "omnimem_allocate launch");
}

omnimem_status omnimem_allocate_noalloc(const omnimem_config* cfg, const omnimem_layer* layers, const float* a,
                                        const float* s, int64_t total_budget, int32_t* budgets, float* stats,
                                        hipStream_t stream) {
  if (!cfg) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null config");
  omnimem_status st = check_config(*cfg);
  if (st != OMNIMEM_OK) return st;
  const Dims dm = make_dims(*cfg);
  const size_t desc_bytes = ((size_t)cfg->n_layers * sizeof(LayerDesc) + 255) / 256 * 256;
  const size_t part_bytes = (size_t)cfg->n_layers * cfg->n_kv_heads * allocate_part_chunks(dm) * 2 * 4 * sizeof(double);
  if (desc_bytes + part_bytes > kScratchBytes)
    return fail(nullptr, OMNIMEM_ERR_CAPACITY, "scratch of %zu bytes needed (layer table %zu + partial sums %zu); "
                "the fixed scratch holds %zu", desc_bytes + part_bytes, desc_bytes, part_bytes, kScratchBytes);
  omnimem_ctx check;  // host-only: argument checks and their message
  check.cfg = *cfg;
  if ((st = check_allocate(&check, layers, a, s, total_budget, budgets)) != OMNIMEM_OK) {
    g_create_error = check.err;
    return st;
  }
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return fail(nullptr, OMNIMEM_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if ((e = hipGetLastError()) != hipSuccess)
    return fail(nullptr, OMNIMEM_ERR_HIP, "earlier device error: %s", hipGetErrorString(e));
  void* base = nullptr;
  if ((st = scratch_address(device, &base)) != OMNIMEM_OK) return st;
  LayerDesc* table = static_cast<LayerDesc*>(base);
  Workspace ws{};
  ws.stat_part = reinterpret_cast<double*>(static_cast<char*>(base) + desc_bytes);
  for (int l0 = 0; l0 < cfg->n_layers; l0 += kDescPerStore) {
    DescBlock blk;
    std::memset(&blk, 0, sizeof blk);
    const int count = std::min(kDescPerStore, cfg->n_layers - l0);
    for (int i = 0; i < count; ++i) describe(*cfg, layers[l0 + i], nullptr, &blk.d[i]);
    store_descs<<<1, 64, 0, stream>>>(table + l0, blk, count);
  }
  e = launch_allocate(dm, table, ws, a, s, total_budget, cfg->ratio_r, cfg->temperature, cfg->b_min_frac,
                      cfg->b_max_frac, budgets, stats, stream);
  if (e != hipSuccess) return fail(nullptr, OMNIMEM_ERR_HIP, "omnimem_allocate_noalloc launch: %s", hipGetErrorString(e));
  g_create_error.clear();
  return OMNIMEM_OK;
}

omnimem_status omnimem_calibrate(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a, const float* s,
                                 float* stats, hipStream_t stream) {
  omnimem_status st = validate(ctx, layers, 0);
  if (st != OMNIMEM_OK) return st;
  if (!a || !s) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null a or s");
  if (ctx->calib_steps == INT32_MAX) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "too many calibration steps");
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  st = finish(ctx, launch_calibrate(ctx->dm, dev, ctx->ws, a, s, ctx->cfg.ratio_r, ctx->calib_steps == 0, stats,
                                    stream),
              stream, "omnimem_calibrate launch");
  if (st == OMNIMEM_OK) ++ctx->calib_steps;
  return st;
}

omnimem_status omnimem_calibration_reset(omnimem_ctx* ctx) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  ctx->calib_steps = 0;
  return OMNIMEM_OK;
}

omnimem_status omnimem_calibration_budgets(omnimem_ctx* ctx, int64_t total_budget, int32_t* layer_budgets,
                                           hipStream_t stream) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  if (!layer_budgets) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null layer_budgets");
  if (ctx->calib_steps == 0) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "no calibration step was added");
  const omnimem_config& c = ctx->cfg;
  if (total_budget < 0 || total_budget > (int64_t)INT32_MAX)
    return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "total budget %lld out of range", (long long)total_budget);
  const int64_t lo_base = (int64_t)std::ceil(((double)c.b_min_frac * (double)total_budget) / c.n_layers);
  if (lo_base * c.n_layers > total_budget)
    return fail(ctx, OMNIMEM_ERR_INFEASIBLE, "per-layer minimum budgets sum to %lld > total %lld",
                (long long)(lo_base * c.n_layers), (long long)total_budget);
  omnimem_status st = set_device(ctx);
  if (st != OMNIMEM_OK) return st;
  return finish(ctx, launch_calibration_budgets(ctx->dm, ctx->ws, total_budget, c.temperature, c.b_min_frac,
                                                c.b_max_frac, ctx->calib_steps, layer_budgets, stream),
                stream, "omnimem_calibration_budgets launch");
}

omnimem_status omnimem_allocate_fixed(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a, const float* s,
                                      const int32_t* layer_budgets, int32_t* budgets, float* stats,
                                      hipStream_t stream) {
  omnimem_status st = validate(ctx, layers, 0);
  if (st != OMNIMEM_OK) return st;
  if (!a || !s || !layer_budgets || !budgets)
    return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null a, s, layer_budgets or budgets");
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  return finish(ctx, launch_allocate_fixed(ctx->dm, dev, ctx->ws, a, s, layer_budgets, ctx->cfg.ratio_r, budgets,
                                           stats, stream),
                stream, "omnimem_allocate_fixed launch");
}

omnimem_status omnimem_select_compact(omnimem_ctx* ctx, const omnimem_layer* layers, const float* a, const float* s,
                                      const int32_t* budgets, int32_t* idx, hipStream_t stream) {
  omnimem_status st = validate(ctx, layers, NEED_K | NEED_V | NEED_OUT);
  if (st != OMNIMEM_OK) return st;
  if (!a || !s || !budgets) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null a, s or budgets");
  bool hidden = false;  // some layer carries its kept rows' hidden states
  if (ctx->cfg.sim_source == OMNIMEM_SRC_HIDDEN) {
    if ((st = validate_hidden(ctx, layers, true)) != OMNIMEM_OK) return st;
    for (int l = 0; l < ctx->cfg.n_layers; ++l) hidden = hidden || layers[l].hidden_out != nullptr;
  }
  int n_inplace = 0;  // layers compacted in place
  for (int l = 0; l < ctx->cfg.n_layers; ++l) n_inplace += in_place(layers[l]) ? 1 : 0;
  const int inplace = n_inplace == 0 ? 0 : n_inplace == ctx->cfg.n_layers ? 2 : 1;
  int64_t max_n = 1;
  for (int l = 0; l < ctx->cfg.n_layers; ++l) max_n = std::max<int64_t>(max_n, layers[l].n_cache + layers[l].n_chunk);
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev)) != OMNIMEM_OK) return st;
  // the ranking path: AUTO by the longest working set; a path that cannot
  // take these sizes falls back to the one-workgroup ranking
  int path = ctx->topk_path;
  if (path == OMNIMEM_TOPK_AUTO)
    path = max_n <= kTopkRegRows ? OMNIMEM_TOPK_REGISTERS
           : max_n > kTopkAutoSplitRows ? OMNIMEM_TOPK_SPLIT : OMNIMEM_TOPK_ONE_WORKGROUP;
  if ((path == OMNIMEM_TOPK_REGISTERS && max_n > kTopkRegRows) ||
      (path == OMNIMEM_TOPK_SPLIT && max_n > kTopkSplitMaxRows))
    path = OMNIMEM_TOPK_ONE_WORKGROUP;
  return finish(ctx, launch_select_compact(ctx->dm, ctx->cfg.dtype, ctx->cfg.lambda, ctx->cfg.shared_selection ? 1 : 0,
                                           hidden, inplace, (int)max_n, path, dev, ctx->ws, a, s, budgets, idx,
                                           stream),
                stream, "omnimem_select_compact launch");
}

omnimem_status omnimem_inplace_status(omnimem_ctx* ctx, int64_t* rows_needed) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  if (rows_needed) *rows_needed = 0;
  omnimem_status st = set_device(ctx);
  if (st != OMNIMEM_OK) return st;
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(ctx, e, "inplace status wait");
  int words[4] = {0, 0, 0, 0};
  if ((e = hipMemcpy(words, ctx->ws.ctl, sizeof words, hipMemcpyDeviceToHost)) != hipSuccess)
    return hip_fail(ctx, e, "inplace status read");
  const int zero[2] = {0, 0};
  if ((e = hipMemcpy(ctx->ws.ctl + 2, zero, sizeof zero, hipMemcpyHostToDevice)) != hipSuccess)
    return hip_fail(ctx, e, "inplace status clear");
  if (rows_needed) *rows_needed = words[2];
  if (words[3] != 0)
    return fail(ctx, OMNIMEM_ERR_HIP, "%d ordering waits of the in-place pass gave up", words[3]);
  if (words[2] != 0)
    return fail(ctx, OMNIMEM_ERR_CAPACITY, "an in-place compaction needed %d staging rows per (layer, KV head); "
                "the context reserves %d: that call moved no row", words[2], ctx->cfg.inplace_stage_rows);
  ctx->err.clear();
  return OMNIMEM_OK;
}

omnimem_status omnimem_append(omnimem_ctx* ctx, const omnimem_layer* layers, const omnimem_chunk* chunks,
                              hipStream_t stream) {
  omnimem_status st = validate(ctx, layers, NEED_K | NEED_V);
  if (st != OMNIMEM_OK) return st;
  if ((st = validate_append(ctx, layers, chunks)) != OMNIMEM_OK) return st;
  int64_t max_rows = 0;
  for (int l = 0; l < ctx->cfg.n_layers; ++l) max_rows = std::max<int64_t>(max_rows, layers[l].n_chunk);
  if ((st = set_device(ctx)) != OMNIMEM_OK) return st;
  const LayerDesc* dev = nullptr;
  if ((st = upload(ctx, layers, stream, &dev, chunks)) != OMNIMEM_OK) return st;
  if (max_rows == 0) return finish(ctx, hipSuccess, stream, "omnimem_append");
  return finish(ctx, launch_append(ctx->dm, ctx->cfg.dtype, dev, ctx->ws, max_rows, stream), stream,
                "omnimem_append launch");
}

omnimem_status omnimem_set_topk_path(omnimem_ctx* ctx, int32_t path) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  if (path < OMNIMEM_TOPK_AUTO || path > OMNIMEM_TOPK_SPLIT)
    return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "top-k path %d is not an omnimem_topk_path", path);
  ctx->topk_path = path;
  return OMNIMEM_OK;
}

omnimem_status omnimem_profile(omnimem_ctx* ctx, int32_t on) {
  if (!ctx) return fail(nullptr, OMNIMEM_ERR_INVALID_ARG, "null context");
  omnimem_status st = set_device(ctx);
  if (st != OMNIMEM_OK) return st;
  if (on && ctx->prof.pool.empty()) {
    ctx->prof.pool.resize(kProfEvents);
    for (auto& e : ctx->prof.pool) {
      // timing only: no system-scope fence (cache writeback and invalidation) at each record,
      // which would slow the kernel that follows it
      hipError_t err = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
      if (err != hipSuccess) return hip_fail(ctx, err, "profiling events");
    }
  }
  ctx->ws.prof = on ? &ctx->prof : nullptr;
  return OMNIMEM_OK;
}

omnimem_status omnimem_profile_report(omnimem_ctx* ctx, omnimem_kernel_time* out, int32_t capacity,
                                      int32_t* count) {
  if (!ctx || (!out && capacity > 0) || !count) return fail(ctx, OMNIMEM_ERR_INVALID_ARG, "null argument");
  omnimem_status st = set_device(ctx);
  if (st != OMNIMEM_OK) return st;
  Profiler& p = ctx->prof;
  double total[K_COUNT] = {};
  int n[K_COUNT] = {};
  int order[K_COUNT];
  int n_kinds = 0;
  for (size_t i = 0; i < p.kernel.size(); ++i) {
    hipError_t e = hipEventSynchronize(p.pool[p.first[i] + 1]);
    if (e != hipSuccess) return hip_fail(ctx, e, "profile wait");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, p.pool[p.first[i]], p.pool[p.first[i] + 1]);
    if (e != hipSuccess) return hip_fail(ctx, e, "profile elapsed time");
    const int k = p.kernel[i];
    if (n[k] == 0) order[n_kinds++] = k;
    n[k] += 1;
    total[k] += ms;
  }
  const int m = std::min<int>(n_kinds, std::max<int32_t>(capacity, 0));
  for (int i = 0; i < m; ++i) {
    const int k = order[i];
    std::memset(&out[i], 0, sizeof out[i]);
    std::snprintf(out[i].name, sizeof out[i].name, "%s", kKernelNames[k]);
    out[i].launches = n[k];
    out[i].total_ms = total[k];
  }
  *count = m;
  p.kernel.clear();
  p.first.clear();
  p.used = 0;
  p.open = false;
  return OMNIMEM_OK;
}

}  // extern "C"
