// C ABI of the keyless-attention library: argument validation, workspace
// sizing, split selection and kernel launches on the caller's stream.
// Nothing here allocates, frees or synchronises.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <string>

#include "keyless.h"
#include "kl_internal.h"

namespace {

thread_local std::string g_err;
thread_local hipEvent_t g_timer_start = nullptr;
thread_local hipEvent_t g_timer_stop = nullptr;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return KL_OK;
  return fail(KL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t elem_bytes(kl_dtype dt) { return dt == KL_BF16 ? 2 : 4; }

bool dtype_ok(kl_dtype dt) { return dt == KL_BF16 || dt == KL_F32; }

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

int log2_exact(int v) {
  if (v <= 0 || (v & (v - 1))) return -1;
  int s = 0;
  while ((1 << s) < v) ++s;
  return s;
}

float scale_or_default(float scale, int d_head) {
  return scale != 0.f ? scale : 1.f / std::sqrt((float)d_head);
}

constexpr float kLog2e = 1.4426950408889634f;

// Validates a cache descriptor. Returns KL_OK or an error code (message set).
int check_cache(const kl_value_cache* c, const char* name) {
  if (!c) return fail(KL_ERR_INVALID_ARG, "%s: descriptor is NULL", name);
  if (!c->data) return fail(KL_ERR_INVALID_ARG, "%s: data is NULL", name);
  if (!aligned16(c->data)) return fail(KL_ERR_INVALID_ARG, "%s: data is not 16-byte aligned", name);
  if (!dtype_ok(c->dtype)) return fail(KL_ERR_UNSUPPORTED, "%s: unknown dtype %d", name, (int)c->dtype);
  if (c->d_head != 64 && c->d_head != 128)
    return fail(KL_ERR_UNSUPPORTED, "%s: d_head %d not supported (64 or 128)", name, c->d_head);
  if (c->G <= 0) return fail(KL_ERR_INVALID_ARG, "%s: G must be positive (got %d)", name, c->G);
  if (c->layout == KL_CONTIGUOUS) {
    if (c->L_max < 0) return fail(KL_ERR_INVALID_ARG, "%s: L_max is negative", name);
  } else if (c->layout == KL_PAGED) {
    if (log2_exact(c->block_size) < 4)
      return fail(KL_ERR_UNSUPPORTED, "%s: block_size %d must be a power of two >= 16", name,
                  c->block_size);
    if (c->num_blocks <= 0 || c->max_blocks_per_seq <= 0)
      return fail(KL_ERR_INVALID_ARG, "%s: num_blocks and max_blocks_per_seq must be positive", name);
    if (!c->block_table) return fail(KL_ERR_INVALID_ARG, "%s: block_table is NULL", name);
    if ((long)c->max_blocks_per_seq * c->block_size > (1L << 30))
      return fail(KL_ERR_UNSUPPORTED, "%s: capacity per sequence too large", name);
  } else {
    return fail(KL_ERR_INVALID_ARG, "%s: unknown layout %d", name, (int)c->layout);
  }
  return KL_OK;
}

int cache_capacity(const kl_value_cache* c) {
  return c->layout == KL_PAGED ? c->max_blocks_per_seq * c->block_size : c->L_max;
}

// Work split of a decode call.
//  - chunk_rows > 0: split mode with that many rows per split (grid S x G x B).
//  - A contiguous cache with at least one (b, g) pair per compute unit: one
//    workgroup per pair streams its whole cache and writes the output directly.
//  - At most kSmallBatch sequences: split mode with splits sized from the
//    capacity (see below).
//  - Otherwise balanced mode: kBalancedWorkgroups workgroups (two per compute
//    unit) take equal shares of the 16-row tiles of all pairs, whatever the
//    spread of lengths, and a merge kernel combines pairs that were shared.
//    Used while the tile count fits comfortably in 32 bits; beyond that the
//    cache is split into chunks of 8192 rows.
struct DecodePlan {
  int chunk, S;
  bool balanced;
};

constexpr int kComputeUnits = 256;
constexpr int kBalancedWorkgroups = 2 * kComputeUnits;
constexpr int kSmallBatch = 4;                        // sequences decoded with fixed splits
constexpr long kSplitWorkgroups = 2 * kComputeUnits;  // their target split count

DecodePlan plan_decode(const kl_value_cache* c, int B, int chunk_rows) {
  const int cap = cache_capacity(c);
  const long pairs = (long)B * c->G;
  DecodePlan pl{};
  if (chunk_rows > 0) {
    pl.chunk = chunk_rows;
  } else if (c->layout == KL_CONTIGUOUS && pairs >= kComputeUnits) {
    pl.chunk = ((cap > 0 ? cap : 1) + 63) / 64 * 64;
  } else if (B <= kSmallBatch && cap > 0) {
    // A few sequences (batch-1 serving): fixed splits, about kSplitWorkgroups
    // of them over the whole capacity and at least 256 rows each; a cache of at
    // most 1024 rows is one split (no merge). Splits past a sequence's length
    // exit at once, so raggedness among so few sequences costs little, and no
    // plan kernel runs.
    const long per = (cap * pairs + kSplitWorkgroups - 1) / kSplitWorkgroups;
    const long chunk = cap <= 1024 ? cap : std::max(256L, per);
    pl.chunk = (int)((chunk + 63) / 64 * 64);
  } else if (pairs * ((long)cap + 15) / 16 < (1L << 30)) {
    pl.balanced = true;
    pl.chunk = 0;
    pl.S = 0;
    return pl;
  } else {
    pl.chunk = 8192;
  }
  pl.S = cap > 0 ? (cap + pl.chunk - 1) / pl.chunk : 1;
  return pl;
}

// Workspace: split partials (acc[d], m, l) per (b, h, split), none with a
// single split; in balanced mode the plan (B + 3 ints) and then one partial row
// per head for each of B * G + kBalancedWorkgroups segment slots.
size_t plan_bytes(int B) { return align256((size_t)(B + 3) * sizeof(int)); }
size_t partials_bytes(const DecodePlan& pl, int B, int H, int G, int d_head) {
  if (pl.balanced)
    return plan_bytes(B) + align256(((size_t)B * G + kBalancedWorkgroups) * (H / G) *
                                    (d_head + 2) * sizeof(float));
  return pl.S > 1 ? align256((size_t)B * H * pl.S * (d_head + 2) * sizeof(float)) : 0;
}

// Query heads per cached group the decode kernels handle.
int check_group_ratio(const char* who, const kl_value_cache* c, int R) {
  const bool wide_groups = c->dtype == KL_BF16 && c->d_head == 128;
  if (!(R >= 1 && R <= 8) && !((R == 16 || R == 32) && wide_groups))
    return fail(KL_ERR_UNSUPPORTED,
                "%s: H/G=%d not supported (1 to 8; also 16 or 32 for bf16 with d_head 128)", who, R);
  return KL_OK;
}

int decode_common(const void* q, const kl_value_cache* k_cache, const kl_value_cache* v_cache,
                  const int32_t* lengths, int B, int H, float scale, void* out, void* ws,
                  size_t ws_bytes, int chunk_rows, void* stream, const char* who,
                  const void* vnew = nullptr) {
  int st = check_cache(v_cache, who);
  if (st != KL_OK) return st;
  if (k_cache) {
    st = check_cache(k_cache, "k_cache");
    if (st != KL_OK) return st;
    if (k_cache->layout != KL_CONTIGUOUS || v_cache->layout != KL_CONTIGUOUS)
      return fail(KL_ERR_UNSUPPORTED, "%s: only contiguous key/value caches", who);
    if (k_cache->dtype != v_cache->dtype || k_cache->G != v_cache->G ||
        k_cache->d_head != v_cache->d_head || k_cache->L_max != v_cache->L_max)
      return fail(KL_ERR_INVALID_ARG, "%s: key and value caches differ in shape or dtype", who);
  }
  if (!q || !lengths || !out)
    return fail(KL_ERR_INVALID_ARG, "%s: q, lengths and out must be non-NULL", who);
  if (!aligned16(q) || !aligned16(out))
    return fail(KL_ERR_INVALID_ARG, "%s: q and out must be 16-byte aligned", who);
  if (B < 0 || H <= 0) return fail(KL_ERR_INVALID_ARG, "%s: bad B=%d or H=%d", who, B, H);
  const int G = v_cache->G;
  if (H % G != 0) return fail(KL_ERR_INVALID_ARG, "%s: H=%d is not a multiple of G=%d", who, H, G);
  const int R = H / G;
  st = check_group_ratio(who, v_cache, R);
  if (st != KL_OK) return st;
  if (chunk_rows < 0 || chunk_rows % 64 != 0)
    return fail(KL_ERR_INVALID_ARG, "%s: chunk_rows=%d must be a multiple of 64", who, chunk_rows);
  if (B == 0) return KL_OK;
  const DecodePlan pl = plan_decode(v_cache, B, chunk_rows);
  if (pl.S > kl::kMaxSplits)
    return fail(KL_ERR_UNSUPPORTED, "%s: %d splits exceed the maximum of %d (use larger chunks)",
                who, pl.S, kl::kMaxSplits);
  const size_t need = partials_bytes(pl, B, H, G, v_cache->d_head);
  if (need && (!ws || ws_bytes < need))
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who, need, ws_bytes);
  if (need && !aligned16(ws))
    return fail(KL_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);

  kl::DecodeParams p{};
  p.q = q;
  p.vdata = v_cache->data;
  p.kdata = k_cache ? k_cache->data : nullptr;
  p.table = v_cache->layout == KL_PAGED ? v_cache->block_table : nullptr;
  p.lengths = lengths;
  p.vnew = vnew;
  p.out = out;
  p.balanced = pl.balanced;
  p.nwg = kBalancedWorkgroups;
  if (pl.balanced) {
    p.plan = static_cast<int*>(ws);
    p.part = reinterpret_cast<float*>(static_cast<char*>(ws) + plan_bytes(B));
  } else {
    p.part = static_cast<float*>(ws);
  }
  p.B = B;
  p.H = H;
  p.G = G;
  p.D = v_cache->d_head;
  p.R = R;
  p.dtype = v_cache->dtype;
  p.paged = v_cache->layout == KL_PAGED;
  p.L_max = v_cache->L_max;
  p.block_shift = p.paged ? log2_exact(v_cache->block_size) : 0;
  p.num_blocks = v_cache->num_blocks;
  p.max_blocks = v_cache->max_blocks_per_seq;
  p.chunk = pl.chunk;
  p.S = pl.S;
  p.scale_log2 = scale_or_default(scale, p.D) * kLog2e;
  p.ev_start = g_timer_start;
  p.ev_stop = g_timer_stop;
  return hip_status(kl::launch_decode(p, static_cast<hipStream_t>(stream)), who);
}

}  // namespace

extern "C" {

const char* keyless_last_error(void) { return g_err.c_str(); }

const char* keyless_version(void) { return "keyless-gfx950 0.1"; }

int keyless_probe_read(const void* src, size_t bytes, unsigned* sink, int workgroups,
                       void* stream) {
  const char* who = "keyless_probe_read";
  if (!src || !sink) return fail(KL_ERR_INVALID_ARG, "%s: src and sink must be non-NULL", who);
  if (bytes % 16 != 0 || !aligned16(src))
    return fail(KL_ERR_INVALID_ARG, "%s: src must be 16-byte aligned and bytes a multiple of 16", who);
  if (workgroups < 1 || workgroups > (1 << 20))
    return fail(KL_ERR_INVALID_ARG, "%s: workgroups=%d outside [1, 2^20]", who, workgroups);
  if (bytes == 0) return KL_OK;
  return hip_status(kl::launch_probe_read(src, bytes, sink, workgroups,
                                          static_cast<hipStream_t>(stream)), who);
}

int keyless_probe_mfma(float* sink, int iters, int workgroups, void* stream) {
  const char* who = "keyless_probe_mfma";
  if (!sink) return fail(KL_ERR_INVALID_ARG, "%s: sink must be non-NULL", who);
  if (iters < 1 || workgroups < 1 || workgroups > (1 << 20))
    return fail(KL_ERR_INVALID_ARG, "%s: iters=%d or workgroups=%d out of range", who, iters,
                workgroups);
  return hip_status(kl::launch_probe_mfma(sink, iters, workgroups, static_cast<hipStream_t>(stream)),
                    who);
}

void keyless_set_kernel_timer(void* start_event, void* stop_event) {
  const bool on = start_event && stop_event;
  g_timer_start = on ? static_cast<hipEvent_t>(start_event) : nullptr;
  g_timer_stop = on ? static_cast<hipEvent_t>(stop_event) : nullptr;
}

size_t keyless_decode_workspace_size(const kl_value_cache* cache, int B, int H, int chunk_rows) {
  if (!cache || B <= 0 || H <= 0 || cache->G <= 0 || chunk_rows < 0) return 0;
  const DecodePlan pl = plan_decode(cache, B, chunk_rows);
  return partials_bytes(pl, B, H, cache->G, cache->d_head);
}

int keyless_decode(const void* q_routed, const kl_value_cache* cache, const int32_t* lengths,
                   int B, int H, float scale, void* out, void* ws, size_t ws_bytes, void* stream) {
  return decode_common(q_routed, nullptr, cache, lengths, B, H, scale, out, ws, ws_bytes, 0,
                       stream, "keyless_decode");
}

int keyless_decode_append(const void* q_routed, const void* v_new, const kl_value_cache* cache,
                          const int32_t* lengths_before, int B, int H, float scale, void* out,
                          void* ws, size_t ws_bytes, void* stream) {
  const char* who = "keyless_decode_append";
  if (!v_new) return fail(KL_ERR_INVALID_ARG, "%s: v_new must be non-NULL", who);
  if (!aligned16(v_new)) return fail(KL_ERR_INVALID_ARG, "%s: v_new must be 16-byte aligned", who);
  return decode_common(q_routed, nullptr, cache, lengths_before, B, H, scale, out, ws, ws_bytes, 0,
                       stream, who, v_new);
}

int keyless_decode_noalloc(const void* q_routed, const kl_value_cache* cache,
                           const int32_t* lengths, int B, int H, float scale, void* out,
                           void* stream) {
  const char* who = "keyless_decode_noalloc";
  int st = check_cache(cache, who);
  if (st != KL_OK) return st;
  if (B < 0 || H <= 0) return fail(KL_ERR_INVALID_ARG, "%s: bad B=%d or H=%d", who, B, H);
  const size_t need = keyless_decode_workspace_size(cache, B, H, 0);
  if (need > kl::kScratchBytes)
    return fail(KL_ERR_UNSUPPORTED,
                "%s: this decode needs %zu bytes of scratch, more than the %zu bytes the "
                "entry point holds; call keyless_decode with a workspace",
                who, need, kl::kScratchBytes);
  void* ws = nullptr;
  if (need > 0 && B > 0) {
    int s = hip_status(kl::scratch_address(&ws), who);
    if (s != KL_OK) return s;
  }
  return decode_common(q_routed, nullptr, cache, lengths, B, H, scale, out, ws,
                       ws ? kl::kScratchBytes : 0, 0, stream, who);
}

int keyless_decode_chunked(const void* q_routed, const kl_value_cache* cache,
                           const int32_t* lengths, int B, int H, float scale, void* out, void* ws,
                           size_t ws_bytes, int chunk_rows, void* stream) {
  return decode_common(q_routed, nullptr, cache, lengths, B, H, scale, out, ws, ws_bytes,
                       chunk_rows, stream, "keyless_decode_chunked");
}

size_t keyless_latent_decode_workspace_size(const kl_value_cache* latent_cache, int B, int H,
                                            int d_head) {
  if (!latent_cache || B <= 0 || H <= 0 || latent_cache->G <= 0 || d_head <= 0) return 0;
  const size_t v = align256((size_t)B * H * latent_cache->d_head * elem_bytes(latent_cache->dtype));
  return 2 * v + keyless_decode_workspace_size(latent_cache, B, H, 0);
}

int keyless_latent_decode(const void* q_routed, const void* W_post,
                          const kl_value_cache* latent_cache, const int32_t* lengths, int B, int H,
                          int d_head, float scale, void* out, void* ws, size_t ws_bytes,
                          void* stream) {
  const char* who = "keyless_latent_decode";
  if (!q_routed || !W_post || !out || !lengths)
    return fail(KL_ERR_INVALID_ARG, "%s: q_routed, W_post, lengths and out must be non-NULL", who);
  if (!aligned16(q_routed) || !aligned16(W_post))
    return fail(KL_ERR_INVALID_ARG, "%s: q_routed and W_post must be 16-byte aligned", who);
  int s = check_cache(latent_cache, who);
  if (s != KL_OK) return s;
  if (d_head != 64 && d_head != 128)
    return fail(KL_ERR_UNSUPPORTED, "%s: d_head %d not supported (64 or 128)", who, d_head);
  if (B < 0 || H <= 0) return fail(KL_ERR_INVALID_ARG, "%s: bad B=%d or H=%d", who, B, H);
  const int G = latent_cache->G;
  if (H % G != 0) return fail(KL_ERR_INVALID_ARG, "%s: H=%d is not a multiple of G=%d", who, H, G);
  s = check_group_ratio(who, latent_cache, H / G);
  if (s != KL_OK) return s;
  if (!(scale >= 0.f)) return fail(KL_ERR_INVALID_ARG, "%s: scale must be >= 0 (0 = 1/sqrt(r))", who);
  if (B == 0) return KL_OK;
  const size_t need = keyless_latent_decode_workspace_size(latent_cache, B, H, d_head);
  if (!ws || ws_bytes < need)
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who, need, ws_bytes);
  if (!aligned16(ws)) return fail(KL_ERR_INVALID_ARG, "%s: workspace must be 16-byte aligned", who);
  const int r = latent_cache->d_head;
  const size_t v = align256((size_t)B * H * r * elem_bytes(latent_cache->dtype));
  char* w = static_cast<char*>(ws);
  hipStream_t st = static_cast<hipStream_t>(stream);
  // q* = q~ W_post^T, the decode of q* over the latent rows (o*), out = o* W_post.
  kl::LatentParams lp{q_routed, W_post, w, B, H, r, d_head, 1, latent_cache->dtype};
  s = hip_status(kl::launch_latent_product(lp, st), who);
  if (s != KL_OK) return s;
  s = decode_common(w, nullptr, latent_cache, lengths, B, H, scale, w + v, w + 2 * v,
                    ws_bytes - 2 * v, 0, stream, who);
  if (s != KL_OK) return s;
  lp = kl::LatentParams{w + v, W_post, out, B, H, r, d_head, 0, latent_cache->dtype};
  return hip_status(kl::launch_latent_product(lp, st), who);
}

int standard_decode(const void* q, const kl_value_cache* k_cache, const kl_value_cache* v_cache,
                    const int32_t* lengths, int B, int H, float scale, void* out, void* ws,
                    size_t ws_bytes, void* stream) {
  if (!k_cache) return fail(KL_ERR_INVALID_ARG, "standard_decode: k_cache is NULL");
  return decode_common(q, k_cache, v_cache, lengths, B, H, scale, out, ws, ws_bytes, 0, stream,
                       "standard_decode");
}

int standard_decode_chunked(const void* q, const kl_value_cache* k_cache,
                            const kl_value_cache* v_cache, const int32_t* lengths, int B, int H,
                            float scale, void* out, void* ws, size_t ws_bytes, int chunk_rows,
                            void* stream) {
  if (!k_cache) return fail(KL_ERR_INVALID_ARG, "standard_decode_chunked: k_cache is NULL");
  return decode_common(q, k_cache, v_cache, lengths, B, H, scale, out, ws, ws_bytes, chunk_rows,
                       stream, "standard_decode_chunked");
}

int value_cache_append(const kl_value_cache* cache, const void* values,
                       const int32_t* lengths_before, int B, int T, void* stream) {
  int st = check_cache(cache, "value_cache_append");
  if (st != KL_OK) return st;
  if (!values || !lengths_before)
    return fail(KL_ERR_INVALID_ARG, "value_cache_append: values and lengths_before must be non-NULL");
  if (!aligned16(values)) return fail(KL_ERR_INVALID_ARG, "value_cache_append: values not 16-byte aligned");
  if (B < 0 || T < 0) return fail(KL_ERR_INVALID_ARG, "value_cache_append: bad B=%d or T=%d", B, T);
  if (B == 0 || T == 0) return KL_OK;
  kl::AppendParams p{};
  p.data = cache->data;
  p.values = values;
  p.lengths_before = lengths_before;
  p.table = cache->layout == KL_PAGED ? cache->block_table : nullptr;
  p.B = B;
  p.T = T;
  p.G = cache->G;
  p.D = cache->d_head;
  p.dtype = cache->dtype;
  p.paged = cache->layout == KL_PAGED;
  p.L_max = cache->L_max;
  p.block_shift = p.paged ? log2_exact(cache->block_size) : 0;
  p.num_blocks = cache->num_blocks;
  p.max_blocks = cache->max_blocks_per_seq;
  return hip_status(kl::launch_append(p, static_cast<hipStream_t>(stream)), "value_cache_append");
}

int keyless_fold_routing(const void* W_Q, const void* W_R, int d_model, int H, int d_head,
                         kl_dtype dtype, void* Wt_Q, void* stream) {
  if (!W_Q || !W_R || !Wt_Q)
    return fail(KL_ERR_INVALID_ARG, "keyless_fold_routing: W_Q, W_R and Wt_Q must be non-NULL");
  if (!dtype_ok(dtype)) return fail(KL_ERR_UNSUPPORTED, "keyless_fold_routing: unknown dtype");
  if (d_model <= 0 || H <= 0 || d_head <= 0)
    return fail(KL_ERR_INVALID_ARG, "keyless_fold_routing: sizes must be positive");
  kl::GemmParams g{};
  g.A = W_Q;
  g.Bm = W_R;
  g.C = Wt_Q;
  g.M = d_model;
  g.N = d_head;
  g.K = d_head;
  g.lda = (long)H * d_head;
  g.ldb = d_head;
  g.ldc = (long)H * d_head;
  g.strideA = d_head;
  g.strideB = (long)d_head * d_head;
  g.strideC = d_head;
  g.batch = H;
  g.dtype = dtype;
  return hip_status(kl::launch_gemm_simple(g, static_cast<hipStream_t>(stream)),
                    "keyless_fold_routing");
}

size_t keyless_packed_weights_size(int d_model, int H, int G, int d_head, kl_dtype dtype) {
  if (d_model <= 0 || H <= 0 || G <= 0 || d_head <= 0 || dtype != KL_BF16) return 0;
  return align256((size_t)(H + G) * d_head * d_model * 2);
}

int keyless_pack_weights(const void* W_Q, const void* W_R, const void* W_V, int d_model, int H,
                         int G, int d_head, kl_dtype dtype, void* packed, void* stream) {
  const char* who = "keyless_pack_weights";
  if (!W_Q || !W_V || !packed)
    return fail(KL_ERR_INVALID_ARG, "%s: W_Q, W_V and packed must be non-NULL", who);
  if (dtype != KL_BF16) return fail(KL_ERR_UNSUPPORTED, "%s: packed weights are bf16 only", who);
  if (d_model <= 0 || H <= 0 || G <= 0 || d_head <= 0 || H % G != 0)
    return fail(KL_ERR_INVALID_ARG, "%s: bad sizes d_model=%d H=%d G=%d d_head=%d", who, d_model,
                H, G, d_head);
  if (d_head != 64 && d_head != 128)
    return fail(KL_ERR_UNSUPPORTED, "%s: d_head %d not supported (64 or 128)", who, d_head);
  if (!aligned16(W_Q) || !aligned16(W_V) || !aligned16(W_R) || !aligned16(packed))
    return fail(KL_ERR_INVALID_ARG, "%s: W_Q, W_R, W_V and packed must be 16-byte aligned", who);
  kl::PackParams pp{};
  pp.W_Q = W_Q;
  pp.W_R = W_R;
  pp.W_V = W_V;
  pp.packed = packed;
  pp.d_model = d_model;
  pp.H = H;
  pp.G = G;
  pp.d_head = d_head;
  pp.N = (H + G) * d_head;
  return hip_status(kl::launch_pack_weights(pp, static_cast<hipStream_t>(stream)), who);
}

size_t keyless_prefill_workspace_size(int B, int N, int d_model, int H, int G, int d_head,
                                      kl_dtype dtype, int has_W_R, int has_q_routed_out,
                                      int has_v_out) {
  return keyless_cross_attention_workspace_size(B, N, N, d_model, H, G, d_head, dtype, has_W_R,
                                                has_q_routed_out, has_v_out);
}

size_t keyless_cross_attention_workspace_size(int B, int N_a, int N_b, int d_model, int H, int G,
                                              int d_head, kl_dtype dtype, int has_W_R,
                                              int has_q_routed_out, int has_v_out) {
  if (B < 0 || N_a < 0 || N_b < 0 || d_model <= 0 || H <= 0 || G <= 0 || d_head <= 0) return 0;
  const size_t e = elem_bytes(dtype);
  size_t n = 0;
  if (dtype == KL_BF16)
    n += keyless_packed_weights_size(d_model, H, G, d_head, dtype);
  else if (has_W_R)
    n += align256((size_t)d_model * H * d_head * e);
  if (!has_q_routed_out) n += align256((size_t)B * N_a * H * d_head * e);
  if (!has_v_out) n += align256((size_t)B * N_b * G * d_head * e);
  return n;
}

}  // extern "C"

namespace {

int check_prefill_args(const char* who, const void* x, const void* W, const void* out, int B,
                       int N, int d_model, int H, int G, int d_head, kl_dtype dtype, float scale) {
  if (!x || !W || !out) return fail(KL_ERR_INVALID_ARG, "%s: inputs and out must be non-NULL", who);
  if (!dtype_ok(dtype)) return fail(KL_ERR_UNSUPPORTED, "%s: unknown dtype", who);
  if (B < 0 || N < 0 || d_model <= 0 || H <= 0 || G <= 0)
    return fail(KL_ERR_INVALID_ARG, "%s: bad sizes B=%d N=%d d_model=%d H=%d G=%d", who, B, N,
                d_model, H, G);
  if (d_head != 64 && d_head != 128)
    return fail(KL_ERR_UNSUPPORTED, "%s: d_head %d not supported (64 or 128)", who, d_head);
  if (H % G != 0) return fail(KL_ERR_INVALID_ARG, "%s: H=%d is not a multiple of G=%d", who, H, G);
  if ((long)B * N > (1L << 30)) return fail(KL_ERR_UNSUPPORTED, "%s: B*N too large", who);
  if (!(scale >= 0.f)) return fail(KL_ERR_INVALID_ARG, "%s: scale must be >= 0 (0 = 1/sqrt(d_head))", who);
  return KL_OK;
}

// Cross-attention adds the value sequence: its length in range, and non-NULL
// unless it is empty.
int check_cross_args(const char* who, const void* xb, int B, int N_b) {
  if (!xb && N_b > 0) return fail(KL_ERR_INVALID_ARG, "%s: xb must be non-NULL", who);
  if (N_b < 0) return fail(KL_ERR_INVALID_ARG, "%s: bad N_b=%d", who, N_b);
  if ((long)B * N_b > (1L << 30)) return fail(KL_ERR_UNSUPPORTED, "%s: B*N_b too large", who);
  return KL_OK;
}

// Attention over the routed queries [B, N, H, d_head] and values [B, Nk, G,
// d_head] (Eq. 2 with the Eq. 4 score; Eq. 14 when the two come from different
// sequences).
int run_attention(const char* who, const void* qr, long q_stride, const void* vv, long v_stride,
                  void* out, int B, int N, int Nk, int H, int G, int d_head, int causal,
                  float scale, kl_dtype dtype, hipStream_t st, float* lse = nullptr,
                  float* out_f32 = nullptr) {
  kl::AttnParams a{};
  a.q = qr;
  a.v = vv;
  a.out = out;
  a.q_stride = q_stride;
  a.v_stride = v_stride;
  a.o_stride = (long)H * d_head;
  a.B = B;
  a.N = N;
  a.Nk = Nk;
  a.H = H;
  a.G = G;
  a.D = d_head;
  a.causal = causal ? 1 : 0;
  a.scale_log2 = scale_or_default(scale, d_head) * kLog2e;
  a.dtype = dtype;
  a.lse = lse;
  a.out_f32 = out_f32;
  // No value rows (an empty X^(b)): the VALU kernel writes the zero rows.
  if (Nk > 0 && kl::attn_bf16_supported(a))
    return hip_status(kl::launch_prefill_attention(a, st), who);
  return hip_status(kl::launch_prefill_attention_simple(a, st), who);
}

// Workspace carve-out shared by the entry points: routed queries and values go
// to the caller's buffers when given, else to the workspace (queries first).
struct QV {
  void* qr;
  void* vv;
};
QV carve_qv(char* w, int B, int N_a, int N_b, int H, int G, int d_head, size_t e,
            void* q_routed_out, void* v_out) {
  QV r{q_routed_out, v_out};
  if (!r.qr) {
    r.qr = w;
    w += align256((size_t)B * N_a * H * d_head * e);
  }
  if (!r.vv) r.vv = w;
  return r;
}

// Checks of the bf16 matrix-core path, made before anything is launched: the
// projection GEMM must handle the shape, and every operand must be 16-byte
// aligned (the GEMM and attention kernels move 16-byte chunks of each).
int check_bf16_path(const char* who, const void* xa, const void* xb, int B, int N_a, int N_b,
                    int d_model, int H, int G, int d_head, const void* out,
                    const void* q_routed_out, const void* v_out, const void* ws) {
  const int NQ = H * d_head, NV = G * d_head;
  const int M = std::max(std::max(B * N_a, B * N_b), 1);
  if (const char* why = kl::gemm_bf16_unsupported(M, NQ + NV, d_model, d_model, NQ, NV))
    return fail(KL_ERR_UNSUPPORTED, "%s: %s (d_model=%d)", who, why, d_model);
  if (!aligned16(xa) || (N_b > 0 && !aligned16(xb)) || !aligned16(out) ||
      !aligned16(q_routed_out) || !aligned16(v_out) || !aligned16(ws))
    return fail(KL_ERR_INVALID_ARG,
                "%s: x, xb, out, q_routed_out, v_out and the workspace must be 16-byte aligned",
                who);
  return KL_OK;
}

// bf16 projections and attention against packed weights, queries from xa
// [B, N_a, d_model], values from xb [B, N_b, d_model]. Self-attention (xa == xb,
// N_a == N_b) projects both in one GEMM launch; cross-attention takes two, the
// value one on the packed rows from H d_head on.
int attend_packed_core(const char* who, const void* xa, const void* xb, const void* packed, int B,
                       int N_a, int N_b, int d_model, int H, int G, int d_head, int causal,
                       float scale, void* out, void* qr, void* vv, hipStream_t st) {
  const int NQ = H * d_head, NV = G * d_head;
  const int Ma = B * N_a, Mb = B * N_b;
  int s = KL_OK;
  if (xa == xb && N_a == N_b) {
    if (Ma > 0)
      s = hip_status(kl::launch_gemm_bf16_packed(xa, Ma, d_model, d_model, packed, NQ + NV, NQ, qr,
                                                 NQ, vv, NV, st),
                     who);
  } else {
    if (Ma > 0)
      s = hip_status(kl::launch_gemm_bf16_packed(xa, Ma, d_model, d_model, packed, NQ, NQ, qr, NQ,
                                                 qr, NQ, st),
                     who);
    if (s == KL_OK && Mb > 0) {
      const void* pv = static_cast<const uint16_t*>(packed) + (size_t)NQ * d_model;
      s = hip_status(kl::launch_gemm_bf16_packed(xb, Mb, d_model, d_model, pv, NV, 0, vv, NV, vv,
                                                 NV, st),
                     who);
    }
  }
  if (s != KL_OK || Ma == 0) return s;
  return run_attention(who, qr, NQ, vv, NV, out, B, N_a, N_b, H, G, d_head, causal, scale, KL_BF16,
                       st);
}

int attend_packed_entry(const char* who, const void* xa, const void* xb, const void* packed, int B,
                        int N_a, int N_b, int d_model, int H, int G, int d_head, int causal,
                        float scale, kl_dtype dtype, void* out, void* q_routed_out, void* v_out,
                        void* ws, size_t ws_bytes, hipStream_t st) {
  if (dtype != KL_BF16) return fail(KL_ERR_UNSUPPORTED, "%s: packed weights are bf16 only", who);
  if (!aligned16(packed))
    return fail(KL_ERR_INVALID_ARG, "%s: the packed weights must be 16-byte aligned", who);
  const size_t e = 2;
  const size_t qbytes = q_routed_out ? 0 : align256((size_t)B * N_a * H * d_head * e);
  const size_t vbytes = v_out ? 0 : align256((size_t)B * N_b * G * d_head * e);
  if (qbytes + vbytes && (!ws || ws_bytes < qbytes + vbytes))
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who,
                qbytes + vbytes, ws_bytes);
  if (B == 0 || (N_a == 0 && N_b == 0)) return KL_OK;
  int s = check_bf16_path(who, xa, xb, B, N_a, N_b, d_model, H, G, d_head, out, q_routed_out,
                          v_out, ws);
  if (s != KL_OK) return s;
  const QV qv = carve_qv(static_cast<char*>(ws), B, N_a, N_b, H, G, d_head, e, q_routed_out, v_out);
  return attend_packed_core(who, xa, xb, packed, B, N_a, N_b, d_model, H, G, d_head, causal, scale,
                            out, qv.qr, qv.vv, st);
}

// Projections and attention from the weights as given: bf16 folds and packs them
// into the workspace and takes the packed path; fp32 runs the VALU kernels.
int attend_entry(const char* who, const void* xa, const void* xb, const void* W_Q,
                 const void* W_R, const void* W_V, int B, int N_a, int N_b, int d_model, int H,
                 int G, int d_head, int causal, float scale, kl_dtype dtype, void* out,
                 void* q_routed_out, void* v_out, void* ws, size_t ws_bytes, hipStream_t st) {
  if (!W_V) return fail(KL_ERR_INVALID_ARG, "%s: W_V must be non-NULL", who);
  const size_t need = keyless_cross_attention_workspace_size(
      B, N_a, N_b, d_model, H, G, d_head, dtype, W_R != nullptr, q_routed_out != nullptr,
      v_out != nullptr);
  if (need && (!ws || ws_bytes < need))
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who, need, ws_bytes);
  if (B == 0 || (N_a == 0 && N_b == 0)) return KL_OK;
  const size_t e = elem_bytes(dtype);
  char* w = static_cast<char*>(ws);
  int s;
  if (dtype == KL_BF16) {
    s = check_bf16_path(who, xa, xb, B, N_a, N_b, d_model, H, G, d_head, out, q_routed_out,
                        v_out, ws);
    if (s != KL_OK) return s;
    void* packed = w;
    w += keyless_packed_weights_size(d_model, H, G, d_head, dtype);
    s = keyless_pack_weights(W_Q, W_R, W_V, d_model, H, G, d_head, dtype, packed, st);
    if (s != KL_OK) return s;
    const QV qv = carve_qv(w, B, N_a, N_b, H, G, d_head, e, q_routed_out, v_out);
    return attend_packed_core(who, xa, xb, packed, B, N_a, N_b, d_model, H, G, d_head, causal,
                              scale, out, qv.qr, qv.vv, st);
  }
  // fp32: VALU kernels on the weights as given.
  const void* Wt = W_Q;
  if (W_R) {
    void* fold = w;
    w += align256((size_t)d_model * H * d_head * e);
    s = keyless_fold_routing(W_Q, W_R, d_model, H, d_head, dtype, fold, st);
    if (s != KL_OK) return s;
    Wt = fold;
  }
  const QV qv = carve_qv(w, B, N_a, N_b, H, G, d_head, e, q_routed_out, v_out);
  const int NQ = H * d_head, NV = G * d_head;
  kl::GemmParams g{};
  g.K = d_model;
  g.lda = d_model;
  g.batch = 1;
  g.dtype = dtype;
  g.A = xa;
  g.M = B * N_a;
  g.Bm = Wt;
  g.C = qv.qr;
  g.N = NQ;
  g.ldb = g.ldc = NQ;
  s = hip_status(kl::launch_gemm_simple(g, st), who);
  if (s != KL_OK) return s;
  g.A = xb;
  g.M = B * N_b;
  g.Bm = W_V;
  g.C = qv.vv;
  g.N = NV;
  g.ldb = g.ldc = NV;
  s = hip_status(kl::launch_gemm_simple(g, st), who);
  if (s != KL_OK || N_a == 0) return s;
  return run_attention(who, qv.qr, NQ, qv.vv, NV, out, B, N_a, N_b, H, G, d_head, causal, scale,
                       dtype, st);
}

}  // namespace

extern "C" {

int keyless_prefill_packed(const void* x, const void* packed, int B, int N, int d_model, int H,
                           int G, int d_head, int causal, float scale, kl_dtype dtype, void* out,
                           void* q_routed_out, void* v_out, void* ws, size_t ws_bytes,
                           void* stream) {
  const char* who = "keyless_prefill_packed";
  int s = check_prefill_args(who, x, packed, out, B, N, d_model, H, G, d_head, dtype, scale);
  if (s != KL_OK) return s;
  return attend_packed_entry(who, x, x, packed, B, N, N, d_model, H, G, d_head, causal, scale,
                             dtype, out, q_routed_out, v_out, ws, ws_bytes,
                             static_cast<hipStream_t>(stream));
}

int keyless_cross_attention_packed(const void* xa, const void* xb, const void* packed, int B,
                                   int N_a, int N_b, int d_model, int H, int G, int d_head,
                                   float scale, kl_dtype dtype, void* out, void* q_routed_out,
                                   void* v_out, void* ws, size_t ws_bytes, void* stream) {
  const char* who = "keyless_cross_attention_packed";
  int s = check_prefill_args(who, xa, packed, out, B, N_a, d_model, H, G, d_head, dtype, scale);
  if (s == KL_OK) s = check_cross_args(who, xb, B, N_b);
  if (s != KL_OK) return s;
  return attend_packed_entry(who, xa, xb, packed, B, N_a, N_b, d_model, H, G, d_head, 0, scale,
                             dtype, out, q_routed_out, v_out, ws, ws_bytes,
                             static_cast<hipStream_t>(stream));
}

int keyless_decode_project(const void* x, const void* packed, int B, int d_model, int H, int G,
                           int d_head, kl_dtype dtype, void* q_routed_out, void* v_out,
                           const kl_value_cache* cache, const int32_t* lengths_before,
                           void* stream) {
  const char* who = "keyless_decode_project";
  if (!x || !packed || !q_routed_out)
    return fail(KL_ERR_INVALID_ARG, "%s: x, packed and q_routed_out must be non-NULL", who);
  if (B < 0 || d_model <= 0 || H <= 0 || G <= 0)
    return fail(KL_ERR_INVALID_ARG, "%s: bad B=%d, d_model=%d, H=%d or G=%d", who, B, d_model, H, G);
  if (H % G != 0) return fail(KL_ERR_INVALID_ARG, "%s: H=%d is not a multiple of G=%d", who, H, G);
  if (d_head != 64 && d_head != 128)
    return fail(KL_ERR_UNSUPPORTED, "%s: d_head %d not supported (64 or 128)", who, d_head);
  if (dtype != KL_BF16) return fail(KL_ERR_UNSUPPORTED, "%s: packed weights are bf16 only", who);
  if (!kl::project_supported(d_model))
    return fail(KL_ERR_UNSUPPORTED, "%s: d_model=%d must be a multiple of 32 and at most 16384",
                who, d_model);
  if (!aligned16(x) || !aligned16(packed))
    return fail(KL_ERR_INVALID_ARG, "%s: x and packed must be 16-byte aligned", who);
  if (cache) {
    int st = check_cache(cache, "cache");
    if (st != KL_OK) return st;
    if (cache->dtype != KL_BF16 || cache->G != G || cache->d_head != d_head)
      return fail(KL_ERR_INVALID_ARG, "%s: cache must be bf16 with G=%d groups of d_head=%d", who,
                  G, d_head);
    if (!lengths_before)
      return fail(KL_ERR_INVALID_ARG, "%s: lengths_before is required with a cache", who);
  }
  if (B == 0) return KL_OK;
  kl::ProjectParams p{};
  p.x = static_cast<const uint16_t*>(x);
  p.Wp = static_cast<const uint16_t*>(packed);
  p.q_out = static_cast<uint16_t*>(q_routed_out);
  p.v_out = static_cast<uint16_t*>(v_out);
  p.B = B;
  p.K = d_model;
  p.N = (H + G) * d_head;
  p.NQ = H * d_head;
  p.G = G;
  p.D = d_head;
  p.ldx = d_model;
  p.ldq = (long)H * d_head;
  p.ldv = (long)G * d_head;
  if (cache) {
    p.cache = static_cast<uint16_t*>(cache->data);
    p.table = cache->layout == KL_PAGED ? cache->block_table : nullptr;
    p.lengths_before = lengths_before;
    p.paged = cache->layout == KL_PAGED;
    p.L_max = cache->L_max;
    p.block_shift = p.paged ? log2_exact(cache->block_size) : 0;
    p.num_blocks = cache->num_blocks;
    p.max_blocks = cache->max_blocks_per_seq;
  }
  return hip_status(kl::launch_project(p, static_cast<hipStream_t>(stream)), who);
}

int keyless_prefill(const void* x, const void* W_Q, const void* W_R, const void* W_V, int B,
                    int N, int d_model, int H, int G, int d_head, int causal, float scale,
                    kl_dtype dtype, void* out, void* q_routed_out, void* v_out, void* ws,
                    size_t ws_bytes, void* stream) {
  const char* who = "keyless_prefill";
  int s = check_prefill_args(who, x, W_Q, out, B, N, d_model, H, G, d_head, dtype, scale);
  if (s != KL_OK) return s;
  return attend_entry(who, x, x, W_Q, W_R, W_V, B, N, N, d_model, H, G, d_head, causal, scale,
                      dtype, out, q_routed_out, v_out, ws, ws_bytes,
                      static_cast<hipStream_t>(stream));
}

int keyless_cross_attention(const void* xa, const void* xb, const void* W_Q, const void* W_R,
                            const void* W_V, int B, int N_a, int N_b, int d_model, int H, int G,
                            int d_head, float scale, kl_dtype dtype, void* out,
                            void* q_routed_out, void* v_out, void* ws, size_t ws_bytes,
                            void* stream) {
  const char* who = "keyless_cross_attention";
  int s = check_prefill_args(who, xa, W_Q, out, B, N_a, d_model, H, G, d_head, dtype, scale);
  if (s == KL_OK) s = check_cross_args(who, xb, B, N_b);
  if (s != KL_OK) return s;
  return attend_entry(who, xa, xb, W_Q, W_R, W_V, B, N_a, N_b, d_model, H, G, d_head, 0, scale,
                      dtype, out, q_routed_out, v_out, ws, ws_bytes,
                      static_cast<hipStream_t>(stream));
}

int keyless_attention_forward(const void* q_routed, const void* v, int B, int N, int H, int G,
                              int d_head, int causal, float scale, kl_dtype dtype, void* out,
                              float* lse, float* out_f32, void* stream) {
  const char* who = "keyless_attention_forward";
  int s = check_prefill_args(who, q_routed, v, out, B, N, 64, H, G, d_head, dtype, scale);
  if (s != KL_OK) return s;
  if (!aligned16(q_routed) || !aligned16(v) || !aligned16(out) || !aligned16(out_f32))
    return fail(KL_ERR_INVALID_ARG, "%s: q_routed, v, out and out_f32 must be 16-byte aligned", who);
  if (B == 0 || N == 0) return KL_OK;
  return run_attention(who, q_routed, (long)H * d_head, v, (long)G * d_head, out, B, N, N, H, G,
                       d_head, causal, scale, dtype, static_cast<hipStream_t>(stream), lse, out_f32);
}

size_t keyless_attention_backward_workspace_size(int B, int N, int H) {
  if (B < 0 || N < 0 || H <= 0) return 0;
  return align256((size_t)B * H * N * sizeof(float));
}

int keyless_attention_backward(const void* q_routed, const void* v, const void* out,
                               const float* out_f32, const void* dout, const float* lse, int B,
                               int N, int H, int G,
                               int d_head, int causal, float scale, kl_dtype dtype, void* dq_routed,
                               void* dv, void* ws, size_t ws_bytes, void* stream) {
  const char* who = "keyless_attention_backward";
  int s = check_prefill_args(who, q_routed, v, out, B, N, 64, H, G, d_head, dtype, scale);
  if (s != KL_OK) return s;
  if (!dout || !lse || !dq_routed || !dv)
    return fail(KL_ERR_INVALID_ARG, "%s: dout, lse, dq_routed and dv must be non-NULL", who);
  if (!aligned16(q_routed) || !aligned16(v) || !aligned16(out) || !aligned16(dout) ||
      !aligned16(dq_routed) || !aligned16(dv))
    return fail(KL_ERR_INVALID_ARG, "%s: tensors must be 16-byte aligned", who);
  const size_t need = keyless_attention_backward_workspace_size(B, N, H);
  if (need && (!ws || ws_bytes < need))
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who, need, ws_bytes);
  if (B == 0 || N == 0) return KL_OK;
  kl::BwdParams p{};
  p.q = q_routed;
  p.v = v;
  p.out = out;
  p.out_f32 = out_f32;
  p.dout = dout;
  p.lse = lse;
  p.Dd = static_cast<float*>(ws);
  p.dq = dq_routed;
  p.dv = dv;
  p.q_stride = p.o_stride = p.dq_stride = (long)H * d_head;
  p.v_stride = p.dv_stride = (long)G * d_head;
  p.B = B;
  p.N = N;
  p.H = H;
  p.G = G;
  p.D = d_head;
  p.causal = causal ? 1 : 0;
  p.scale = scale_or_default(scale, d_head);
  p.scale_log2 = p.scale * kLog2e;
  p.dtype = dtype;
  return hip_status(kl::launch_attention_backward(p, static_cast<hipStream_t>(stream)), who);
}

namespace {

// Workspace of the matrix-core form of keyless_weight_gradients (bf16):
// dQ = dQ~ W^R^T [M, H d_head]; the transposes X^T and [dQ^T ; dV^T] over the
// padded token count Mp (the second buffer later holds Q = X W^Q); dQ~^T and
// Q^T [H d_head, Mp]; W^Q^T [H d_head, d_model]; the fp32 partial sums of
// dW^R over S token chunks [S, H, d_head, d_head].
struct WgradLayout {
  long S;   // token chunks of the dW^R contraction (each on its own workgroups)
  long Mp;  // tokens padded to a multiple of 64 S
  size_t dQ, xT, dT, dqT, QT, WQT, part, total;
};

WgradLayout wgrad_layout(long M, long d_model, long NQ, long NV, long H, long dk) {
  WgradLayout L{};
  // dW^R has H d_head x d_head outputs: one workgroup per head would leave
  // most of the chip idle over a long contraction, so the tokens are split.
  L.S = std::max(1L, std::min({16L, 256 / H, (M + 255) / 256}));
  L.Mp = (M + 64 * L.S - 1) / (64 * L.S) * (64 * L.S);
  L.dQ = 0;
  L.xT = L.dQ + align256((size_t)M * NQ * 2);
  L.dT = L.xT + align256((size_t)d_model * L.Mp * 2);
  L.dqT = L.dT + align256((size_t)(NQ + NV) * L.Mp * 2);
  L.QT = L.dqT + align256((size_t)NQ * L.Mp * 2);
  L.WQT = L.QT + align256((size_t)NQ * L.Mp * 2);
  L.part = L.WQT + align256((size_t)NQ * d_model * 2);
  L.total = L.part + align256((size_t)L.S * H * dk * dk * 4);
  return L;
}

}  // namespace

size_t keyless_weight_gradients_workspace_size(int B, int N, int d_model, int H, int G,
                                               int d_head, kl_dtype dtype) {
  if (B < 0 || N < 0 || d_model <= 0 || H <= 0 || G <= 0 || d_head <= 0) return 0;
  const long M = (long)B * N, NQ = (long)H * d_head, NV = (long)G * d_head;
  const size_t generic = 2 * align256((size_t)M * NQ * elem_bytes(dtype));
  if (dtype != KL_BF16) return generic;
  return std::max(generic, wgrad_layout(M, d_model, NQ, NV, H, d_head).total);
}

int keyless_weight_gradients(const void* x, const void* W_Q, const void* W_R, const void* W_V,
                             const void* dq_routed, const void* dv, int B, int N, int d_model,
                             int H, int G, int d_head, kl_dtype dtype, void* dW_Q, void* dW_R,
                             void* dW_V, void* dx, void* ws, size_t ws_bytes, void* stream) {
  const char* who = "keyless_weight_gradients";
  if (!x || !W_Q || !W_R || !W_V || !dq_routed || !dv)
    return fail(KL_ERR_INVALID_ARG, "%s: x, the weights, dq_routed and dv must be non-NULL", who);
  if (!dtype_ok(dtype)) return fail(KL_ERR_UNSUPPORTED, "%s: unknown dtype", who);
  if (B < 0 || N < 0 || d_model <= 0 || H <= 0 || G <= 0 || d_head <= 0)
    return fail(KL_ERR_INVALID_ARG, "%s: bad sizes", who);
  if (H % G != 0) return fail(KL_ERR_INVALID_ARG, "%s: H=%d is not a multiple of G=%d", who, H, G);
  if ((long)B * N > (1L << 30)) return fail(KL_ERR_UNSUPPORTED, "%s: B*N too large", who);
  const size_t need = keyless_weight_gradients_workspace_size(B, N, d_model, H, G, d_head, dtype);
  if (!ws || ws_bytes < need)
    return fail(KL_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", who, need, ws_bytes);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const long M = (long)B * N, NQ = (long)H * d_head, NV = (long)G * d_head;
  char* w = static_cast<char*>(ws);
  auto gemm = [&](const void* A, long lda, long a_cs, const void* Bm, long ldb, long b_cs, void* C,
                  long ldc, long Mm, long Nn, long Kk, int batch, long sA, long sB, long sC,
                  int accumulate) {
    kl::GemmParams g{};
    g.A = A;
    g.Bm = Bm;
    g.C = C;
    g.M = (int)Mm;
    g.N = (int)Nn;
    g.K = (int)Kk;
    g.lda = lda;
    g.a_cs = a_cs;
    g.ldb = ldb;
    g.b_cs = b_cs;
    g.ldc = ldc;
    g.batch = batch;
    g.strideA = sA;
    g.strideB = sB;
    g.strideC = sC;
    g.dtype = dtype;
    g.accumulate = accumulate;
    return hip_status(kl::launch_gemm_simple(g, st), who);
  };
  const long dk = d_head;
  // bf16 with 16-byte aligned operands, head widths and d_model multiples of
  // 64: every product runs on the matrix cores, in the form above (each
  // intermediate, Q = X W^Q and dQ, rounded to bf16 once, as in the generic
  // form; fp32 accumulation). The GEMM takes both operands with the
  // contraction index contiguous, so X, dQ, dV, dQ~ and W^Q are transposed
  // where a product needs it (the token count padded with zeros to a multiple
  // of 64); the per-head products are batched over the heads.
  const WgradLayout L = wgrad_layout(M, d_model, NQ, NV, H, dk);
  const size_t lim = size_t(1) << 32;  // the GEMM's 32-bit operand offsets
  const bool fits = (size_t)d_model * L.Mp * 2 < lim && (size_t)(NQ + NV) * L.Mp * 2 < lim &&
                    (size_t)M * (NQ + NV + d_model) * 2 < lim && (size_t)d_model * (NQ + NV) * 2 < lim;
  if (dtype == KL_BF16 && M > 0 && dk % 64 == 0 && d_model % 64 == 0 && fits && aligned16(x) &&
      aligned16(W_Q) && aligned16(W_R) && aligned16(W_V) && aligned16(dq_routed) && aligned16(dv) &&
      aligned16(ws)) {
    void* dQm = w + L.dQ;   // [M, NQ]
    void* xT = w + L.xT;    // [d_model, Mp]
    char* dT = w + L.dT;    // [NQ + NV, Mp]: dQ^T then dV^T
    void* dqT = w + L.dqT;  // [NQ, Mp]
    void* QT = w + L.QT;    // [NQ, Mp]
    void* WQT = w + L.WQT;  // [NQ, d_model]
    float* part = reinterpret_cast<float*>(w + L.part);  // [S, H, dk, dk]
    int s = KL_OK;
    auto mm = [&](const kl::GemmBf16Args& a) {
      if (const char* why = kl::gemm_bf16_unsupported(a))
        return fail(KL_ERR_UNSUPPORTED, "%s: %s", who, why);
      return hip_status(kl::launch_gemm_bf16(a, st), who);
    };
    auto tr = [&](const void* src, long ld_src, long rows, long cols, void* dst, long ld_dst,
                  long rows_pad) {
      return hip_status(kl::launch_transpose_bf16(src, ld_src, (int)rows, (int)cols, dst, ld_dst,
                                                  (int)rows_pad, st),
                        who);
    };
    // C (rows x cols) = A W^T over K, optionally batched over the heads (item
    // strides sA, sW, sC), columns below n_split to C0, the rest to C1.
    auto prod = [&](const void* A, long lda, long sA, const void* W, long ldw, long sW, long K,
                    long rows, long cols, void* C0, long ldc0, long sC, long n_split, void* C1,
                    long ldc1, int batch) {
      kl::GemmBf16Args a{};
      a.A0 = A;
      a.lda0 = lda;
      a.W0 = W;
      a.ldw0 = ldw;
      a.K0 = (int)K;
      a.M = (int)rows;
      a.N = (int)cols;
      a.n_split = (int)n_split;
      a.C0 = C0;
      a.ldc0 = ldc0;
      a.C1 = C1;
      a.ldc1 = ldc1;
      a.batch = batch;
      a.sA0 = sA;
      a.sW0 = sW;
      a.sC0 = sC;
      a.sC1 = sC;
      return mm(a);
    };
    // dQ_h = dQ~_h W^R_h^T (W^R_h as stored is the [n][k] operand).
    if (dW_Q || dx)
      s = prod(dq_routed, NQ, dk, W_R, dk, dk * dk, dk, M, dk, dQm, NQ, dk, dk, dQm, NQ, H);
    if (s == KL_OK && (dW_Q || dW_V)) {
      // [dW^Q | dW^V] = X^T [dQ | dV], a contraction over the (padded) tokens.
      s = tr(x, d_model, M, d_model, xT, L.Mp, L.Mp);
      if (s == KL_OK && dW_Q) s = tr(dQm, NQ, M, NQ, dT, L.Mp, L.Mp);
      if (s == KL_OK && dW_V) s = tr(dv, NV, M, NV, dT + (size_t)NQ * L.Mp * 2, L.Mp, L.Mp);
      if (s == KL_OK) {
        const char* Wt = dW_Q ? dT : dT + (size_t)NQ * L.Mp * 2;
        const long cols = (dW_Q ? NQ : 0) + (dW_V ? NV : 0);
        s = prod(xT, L.Mp, 0, Wt, L.Mp, 0, L.Mp, d_model, cols, dW_Q ? dW_Q : dW_V,
                 dW_Q ? NQ : NV, 0, dW_Q ? NQ : cols, dW_V ? dW_V : dW_Q, NV, 1);
      }
    }
    if (s == KL_OK && dW_R) {
      // Q = X W^Q (into the [dQ^T ; dV^T] buffer, whose product above has run:
      // the stream orders them), Q^T and dQ~^T with zero token padding, then
      // Eq. 5: dW^R_h = Q_h^T dQ~_h, a contraction over the tokens batched over
      // the heads.
      void* Qm = dT;  // [M, NQ]
      s = tr(W_Q, NQ, d_model, NQ, WQT, d_model, d_model);
      if (s == KL_OK)
        s = prod(x, d_model, 0, WQT, d_model, 0, d_model, M, NQ, Qm, NQ, 0, NQ, Qm, NQ, 1);
      if (s == KL_OK) s = tr(Qm, NQ, M, NQ, QT, L.Mp, L.Mp);
      if (s == KL_OK) s = tr(dq_routed, NQ, M, NQ, dqT, L.Mp, L.Mp);
      if (s == KL_OK) {
        // Item (h, z): rows of head h, tokens of chunk z; fp32 partials, then
        // their sum in chunk order.
        const long Kc = L.Mp / L.S;
        kl::GemmBf16Args a{};
        a.A0 = QT;
        a.lda0 = L.Mp;
        a.W0 = dqT;
        a.ldw0 = L.Mp;
        a.K0 = (int)Kc;
        a.M = (int)dk;
        a.N = (int)dk;
        a.n_split = (int)dk;
        a.C0 = part;
        a.ldc0 = dk;
        a.C1 = part;
        a.ldc1 = dk;
        a.batch = H;
        a.sA0 = dk * L.Mp;
        a.sW0 = dk * L.Mp;
        a.sC0 = dk * dk;
        a.sC1 = dk * dk;
        a.zbatch = (int)L.S;
        a.zA0 = Kc;
        a.zW0 = Kc;
        a.zC0 = H * dk * dk;
        a.c_f32 = 1;
        s = mm(a);
        if (s == KL_OK)
          s = hip_status(kl::launch_sum_partials_bf16(part, (int)L.S, (size_t)H * dk * dk, dW_R, st),
                         who);
      }
    }
    if (s == KL_OK && dx) {
      // dx = dQ W^Q^T + dV W^V^T in one k loop (W^Q, W^V as stored are the
      // [n][k] operands).
      kl::GemmBf16Args a{};
      a.A0 = dQm;
      a.lda0 = NQ;
      a.W0 = W_Q;
      a.ldw0 = NQ;
      a.K0 = (int)NQ;
      a.A1 = dv;
      a.lda1 = NV;
      a.W1 = W_V;
      a.ldw1 = NV;
      a.K1 = (int)NV;
      a.M = (int)M;
      a.N = d_model;
      a.n_split = d_model;
      a.C0 = dx;
      a.ldc0 = d_model;
      a.C1 = dx;
      a.ldc1 = d_model;
      s = mm(a);
    }
    return s;
  }
  // The generic form. With no tokens (M = 0) the contractions over tokens have
  // K = 0 and write zero weight gradients; the token-shaped outputs are empty.
  void* Q = w;                                                   // X W^Q       [M, NQ]
  void* dQ = w + align256((size_t)M * NQ * elem_bytes(dtype));    // dQ~ W^R^T   [M, NQ]
  int s = KL_OK;
  // dQ_h = dQ~_h (W^R_h)^T: B(k, n) = W^R_h[n][k].
  if (dW_Q || dx) s = gemm(dq_routed, NQ, 1, W_R, 1, dk, dQ, NQ, M, dk, dk, H, dk, dk * dk, dk, 0);
  // Eq. 5: dW^R_h = (X W^Q_h)^T dQ~_h, a contraction over the tokens.
  if (s == KL_OK && dW_R) {
    s = gemm(x, d_model, 1, W_Q, NQ, 1, Q, NQ, M, NQ, d_model, 1, 0, 0, 0, 0);
    if (s == KL_OK) s = gemm(Q, 1, NQ, dq_routed, NQ, 1, dW_R, dk, dk, dk, M, H, dk, dk, dk * dk, 0);
  }
  // dW^Q = X^T dQ, and Eq. 6: dW^V = X^T dV (both of its terms are inside dV).
  if (s == KL_OK && dW_Q) s = gemm(x, 1, d_model, dQ, NQ, 1, dW_Q, NQ, d_model, NQ, M, 1, 0, 0, 0, 0);
  if (s == KL_OK && dW_V) s = gemm(x, 1, d_model, dv, NV, 1, dW_V, NV, d_model, NV, M, 1, 0, 0, 0, 0);
  // dX = dQ (W^Q)^T + dV (W^V)^T.
  if (s == KL_OK && dx) {
    s = gemm(dQ, NQ, 1, W_Q, 1, NQ, dx, d_model, M, d_model, NQ, 1, 0, 0, 0, 0);
    if (s == KL_OK) s = gemm(dv, NV, 1, W_V, 1, NV, dx, d_model, M, d_model, NV, 1, 0, 0, 0, 1);
  }
  return s;
}

}  // extern "C"
