// C ABI of libhswa: argument validation, layer-kind dispatch and host helpers.
// Every device call validates synchronously, then enqueues its kernels on the
// caller's stream; nothing here allocates device memory.
#include <cmath>
#include <cstdlib>
#include <cstring>

#include "../../include/hswa.h"
#include "hswa_launch.h"

namespace {

bool sync_check_enabled() {
  static const bool on = [] {
    const char *e = std::getenv("HSWA_SYNC_CHECK");
    return e && e[0] && std::strcmp(e, "0") != 0;
  }();
  return on;
}

hswa_status finish_launch(hipError_t e, hipStream_t stream) {
  if (e != hipSuccess) return HSWA_ERR_LAUNCH;
  if (sync_check_enabled() && hipStreamSynchronize(stream) != hipSuccess) return HSWA_ERR_LAUNCH;
  return HSWA_OK;
}

int log2_exact(int32_t x) {
  if (x <= 0 || (x & (x - 1)) != 0) return -1;
  int s = 0;
  while ((1 << s) < x) ++s;
  return s;
}

constexpr int32_t kMaxKvHeads = 4096;

// Shape checks shared by every device call.
hswa_status check_shape(const hswa_shape *sh) {
  if (!sh) return HSWA_ERR_INVALID_ARG;
  if (sh->num_q_heads <= 0 || sh->num_kv_heads <= 0 || sh->page_size <= 0 || sh->head_dim <= 0)
    return HSWA_ERR_INVALID_ARG;
  if (sh->num_q_heads % sh->num_kv_heads != 0) return HSWA_ERR_INVALID_ARG;
  if (!(sh->scale > 0.f) || !std::isfinite(sh->scale)) return HSWA_ERR_INVALID_ARG;
  if (sh->head_dim != hswa::kHeadDim) return HSWA_ERR_UNSUPPORTED;
  // a page-head of every KV head (Hkv * PG * D * 2 bytes) stays under 2^32,
  // which the kernels' 32-bit page strides assume
  if (sh->num_kv_heads > kMaxKvHeads) return HSWA_ERR_UNSUPPORTED;
  const int group = sh->num_q_heads / sh->num_kv_heads;
  if (128 % group != 0) return HSWA_ERR_UNSUPPORTED;
  const int s = log2_exact(sh->page_size);
  if (s < 4 || s > 8) return HSWA_ERR_UNSUPPORTED;
  return HSWA_OK;
}

hswa_status check_layer(hswa_layer layer) {
  if (layer.kind == HSWA_LAYER_FULL) return HSWA_OK;
  if (layer.kind == HSWA_LAYER_SWA || layer.kind == HSWA_LAYER_SWA_PAGED)
    return layer.window >= 1 ? HSWA_OK : HSWA_ERR_INVALID_ARG;
  return HSWA_ERR_INVALID_ARG;
}

// Builds the kernels' pool view; checks the pieces every call needs.
hswa_status make_pool(hswa_layer layer, const hswa_shape *sh, const hswa_cache *cache, hswa::PoolView &pv) {
  if (!cache || !cache->k_pool || !cache->v_pool || !cache->block_table) return HSWA_ERR_INVALID_ARG;
  if (cache->num_pages <= 0 || cache->table_stride <= 0) return HSWA_ERR_INVALID_ARG;
  pv.k_pool = static_cast<uint16_t *>(cache->k_pool);
  pv.v_pool = static_cast<uint16_t *>(cache->v_pool);
  pv.num_pages = cache->num_pages;
  pv.table = cache->block_table;
  pv.stride = cache->table_stride;
  pv.pg_shift = log2_exact(sh->page_size);
  pv.vb_shift = pv.pg_shift < hswa::kVBlockShiftMax ? pv.pg_shift : hswa::kVBlockShiftMax;
  if (layer.kind == HSWA_LAYER_SWA) {
    pv.ring = hswa_ring_pages(layer.window, sh->page_size);
    pv.window = layer.window;
    if (pv.ring > cache->table_stride) return HSWA_ERR_CAPACITY;
  } else if (layer.kind == HSWA_LAYER_SWA_PAGED) {  // FULL-style table, window masking
    pv.ring = 0;
    pv.window = layer.window;
  } else {
    pv.ring = 0;
    pv.window = 0;
  }
  return HSWA_OK;
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct DecodeGeometry {
  int32_t split_len;
  int32_t max_splits;
  size_t o_bytes;
  size_t total_bytes;
};

constexpr int32_t kMaxQueries = 64;  // queries per sequence in one decode call

// The first of nq new queries of an SWA layer reads the W - 1 keys before it,
// which must still be held once all nq tokens are appended. A ring keeps the
// latest R * PG positions, so nq <= R * PG - W + 1. An explicit-release table
// stores only the last W of the positions one extend adds, so nq <= W.
hswa_status check_multi_window(hswa_layer layer, const hswa_shape *sh, int32_t nq) {
  if (layer.kind == HSWA_LAYER_SWA) {
    const int64_t held = (int64_t)hswa_ring_pages(layer.window, sh->page_size) * sh->page_size;
    if ((int64_t)nq > held - layer.window + 1) return HSWA_ERR_UNSUPPORTED;
  } else if (layer.kind == HSWA_LAYER_SWA_PAGED) {
    if (nq > layer.window) return HSWA_ERR_UNSUPPORTED;
  }
  return HSWA_OK;
}

DecodeGeometry decode_geometry(const hswa_shape *sh, int32_t ns, int32_t max_ctx, int32_t nq) {
  DecodeGeometry g{};
  const int group = sh->num_q_heads / sh->num_kv_heads;
  g.split_len = hswa::decode_split_len(ns, sh->num_kv_heads, group, max_ctx);
  if (max_ctx <= g.split_len) {  // single pass, no workspace
    g.max_splits = 1;
    return g;
  }
  // a segment of at most max_ctx keys meets at most ceil(max_ctx / split_len) + 1
  // spans of at least split_len keys
  g.max_splits = (max_ctx + g.split_len - 1) / g.split_len + 1;
  const size_t rows = (size_t)ns * nq * sh->num_q_heads * g.max_splits;
  g.o_bytes = align_up(rows * sh->head_dim * sizeof(float), 256);
  g.total_bytes = g.o_bytes + align_up(rows * sizeof(float), 256);
  return g;
}

}  // namespace

extern "C" {

int32_t hswa_ring_pages(int32_t window, int32_t page_size) {
  if (window < 1 || page_size < 1) return -1;
  return (int32_t)(((int64_t)window + page_size - 1) / page_size + 1);
}

int64_t hswa_page_bytes(const hswa_shape *shape) {
  if (!shape || shape->num_kv_heads <= 0 || shape->page_size <= 0 || shape->head_dim <= 0) return -1;
  return (int64_t)shape->num_kv_heads * shape->page_size * shape->head_dim * 2;
}

hswa_status hswa_build_block_table(hswa_layer layer, int32_t page_size, int32_t ns, const int32_t *final_lens,
                                   const int32_t *perm, int64_t perm_len, int32_t *table_out, int32_t stride) {
  if (check_layer(layer) != HSWA_OK || page_size < 1 || ns < 0 || stride < 1 || perm_len < 0)
    return HSWA_ERR_INVALID_ARG;
  if (ns > 0 && (!final_lens || !table_out)) return HSWA_ERR_INVALID_ARG;
  if (perm_len > 0 && !perm) return HSWA_ERR_INVALID_ARG;
  int64_t off = 0;
  for (int32_t b = 0; b < ns; ++b) {
    if (final_lens[b] < 0) return HSWA_ERR_INVALID_ARG;
    const int64_t need = layer.kind == HSWA_LAYER_SWA ? hswa_ring_pages(layer.window, page_size)
                                                      : ((int64_t)final_lens[b] + page_size - 1) / page_size;
    if (need > stride || off + need > perm_len) return HSWA_ERR_CAPACITY;
    int32_t *row = table_out + (int64_t)b * stride;
    for (int64_t i = 0; i < stride; ++i) row[i] = i < need ? perm[off + i] : -1;
    off += need;
  }
  return HSWA_OK;
}

hswa_status hswa_kv_append(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *k_new,
                           const void *v_new, const int32_t *cu_seqlens, const int32_t *start_pos, int32_t ns,
                           int32_t total_tokens, int64_t *slot_mapping_out, void *stream) {
  hswa_status st;
  if ((st = check_layer(layer)) != HSWA_OK) return st;
  if ((st = check_shape(shape)) != HSWA_OK) return st;
  if (ns < 0 || total_tokens < 0) return HSWA_ERR_INVALID_ARG;
  hswa::PoolView pv{};
  if ((st = make_pool(layer, shape, cache, pv)) != HSWA_OK) return st;
  if (ns == 0 || total_tokens == 0) return HSWA_OK;
  if (!k_new || !v_new || !cu_seqlens || !start_pos) return HSWA_ERR_INVALID_ARG;
  hswa::AppendParams p{};
  p.pool = pv;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.cu_seqlens = cu_seqlens;
  p.start_pos = start_pos;
  p.slot_out = slot_mapping_out;
  p.ns = ns;
  p.total_tokens = total_tokens;
  p.hkv = shape->num_kv_heads;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return finish_launch(hswa::launch_kv_append(p, s), s);
}

hswa_status hswa_prefill(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                         const void *k_new, const void *v_new, const int32_t *cu_seqlens, const int32_t *prefix_lens,
                         int32_t ns, int32_t total_tokens, int32_t max_chunk_len, void *out, void *stream) {
  hswa_status st;
  if ((st = check_layer(layer)) != HSWA_OK) return st;
  if ((st = check_shape(shape)) != HSWA_OK) return st;
  if (ns < 0 || total_tokens < 0 || max_chunk_len < 0) return HSWA_ERR_INVALID_ARG;
  hswa::PoolView pv{};
  if ((st = make_pool(layer, shape, cache, pv)) != HSWA_OK) return st;
  if (ns == 0 || total_tokens == 0 || max_chunk_len == 0) return HSWA_OK;
  if (!q || !k_new || !v_new || !cu_seqlens || !prefix_lens || !out) return HSWA_ERR_INVALID_ARG;
  hswa::PrefillParams p{};
  p.pool = pv;
  p.q = static_cast<const uint16_t *>(q);
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.cu_seqlens = cu_seqlens;
  p.prefix_lens = prefix_lens;
  p.out = static_cast<uint16_t *>(out);
  p.ns = ns;
  p.total_tokens = total_tokens;
  p.max_chunk_len = max_chunk_len;
  p.hq = shape->num_q_heads;
  p.hkv = shape->num_kv_heads;
  p.group = p.hq / p.hkv;
  p.scale_log2 = shape->scale * 1.4426950408889634f;
  hipStream_t s = static_cast<hipStream_t>(stream);
  return finish_launch(hswa::launch_prefill(p, s), s);
}

size_t hswa_decode_multi_workspace_bytes(const hswa_shape *shape, int32_t ns, int32_t num_queries,
                                         int32_t max_context_len) {
  if (check_shape(shape) != HSWA_OK || ns < 0 || max_context_len < 1) return 0;
  if (num_queries < 1 || num_queries > kMaxQueries) return 0;
  if (ns == 0) return 0;
  return decode_geometry(shape, ns, max_context_len, num_queries).total_bytes;
}

size_t hswa_decode_workspace_bytes(const hswa_shape *shape, int32_t ns, int32_t max_context_len) {
  return hswa_decode_multi_workspace_bytes(shape, ns, 1, max_context_len);
}

int32_t hswa_decode_split_len(const hswa_shape *shape, int32_t ns, int32_t max_context_len) {
  if (check_shape(shape) != HSWA_OK || ns < 1 || max_context_len < 1) return -1;
  return decode_geometry(shape, ns, max_context_len, 1).split_len;
}

}  // extern "C"

namespace {

// Shared body of the decode entry points. With `noalloc` the FULL split
// partials go to the library's fixed device array instead of `workspace`.
// With k_new / v_new (one query per sequence) the call first stores the step's
// new token of every sequence, in the same launch when the kernel allows it.
hswa_status decode_impl(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                        const int32_t *context_lens, int32_t ns, int32_t num_queries, int32_t max_context_len,
                        void *workspace, size_t workspace_bytes, bool noalloc, void *out, void *stream,
                        const void *k_new = nullptr, const void *v_new = nullptr, bool append = false) {
  hswa_status st;
  if ((st = check_layer(layer)) != HSWA_OK) return st;
  if ((st = check_shape(shape)) != HSWA_OK) return st;
  if (ns < 0 || max_context_len < 1 || num_queries < 1 || num_queries > kMaxQueries) return HSWA_ERR_INVALID_ARG;
  hswa::PoolView pv{};
  if ((st = make_pool(layer, shape, cache, pv)) != HSWA_OK) return st;
  if ((st = check_multi_window(layer, shape, num_queries)) != HSWA_OK) return st;
  // FULL-style tables are indexed by the logical page of every position
  if ((layer.kind == HSWA_LAYER_FULL || layer.kind == HSWA_LAYER_SWA_PAGED) &&
      (int64_t)cache->table_stride * shape->page_size < (int64_t)max_context_len)
    return HSWA_ERR_CAPACITY;
  if (ns == 0) return HSWA_OK;
  if (!q || !context_lens || !out) return HSWA_ERR_INVALID_ARG;
  if (append && (!k_new || !v_new)) return HSWA_ERR_INVALID_ARG;
  hswa::DecodeParams p{};
  p.pool = pv;
  p.q = static_cast<const uint16_t *>(q);
  p.ctx_lens = context_lens;
  p.out = static_cast<uint16_t *>(out);
  p.ns = ns;
  p.hq = shape->num_q_heads;
  p.hkv = shape->num_kv_heads;
  p.group = p.hq / p.hkv;
  p.max_ctx = max_context_len;
  p.nq = num_queries;
  p.scale_log2 = shape->scale * 1.4426950408889634f;
  if (layer.kind == HSWA_LAYER_FULL) {
    const DecodeGeometry geo = decode_geometry(shape, ns, max_context_len, num_queries);
    p.split_len = geo.split_len;
    p.max_splits = geo.max_splits;
    if (geo.max_splits > 1) {
      if (noalloc) {
        if (geo.total_bytes > HSWA_NOALLOC_SCRATCH_BYTES) return HSWA_ERR_CAPACITY;
        if (hswa::noalloc_scratch(&workspace) != hipSuccess) return HSWA_ERR_LAUNCH;
      } else {
        if (!workspace) return HSWA_ERR_INVALID_ARG;
        if (workspace_bytes < geo.total_bytes) return HSWA_ERR_CAPACITY;
      }
      p.ws_o = static_cast<float *>(workspace);
      p.ws_lse = reinterpret_cast<float *>(static_cast<char *>(workspace) + geo.o_bytes);
    }
  } else {
    p.split_len = max_context_len;
    p.max_splits = 1;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (append) {
    p.k_new = static_cast<const uint16_t *>(k_new);
    p.v_new = static_cast<const uint16_t *>(v_new);
    if (hswa::decode_append_fused(p)) return finish_launch(hswa::launch_decode_append(p, s), s);
    if (p.max_splits > 1 && p.nq == 1 && pv.pg_shift >= 5) {
      // FULL split path: the split decode stores the token itself
      p.split_append = 1;
      return finish_launch(hswa::launch_decode(p, s), s);
    }
    hswa::AppendParams a{};
    a.pool = pv;
    a.k_new = p.k_new;
    a.v_new = p.v_new;
    a.ns = ns;
    a.total_tokens = ns;
    a.hkv = p.hkv;
    a.ctx_lens = context_lens;
    a.max_ctx = max_context_len;
    const hipError_t e = hswa::launch_kv_append(a, s);
    if (e != hipSuccess) return HSWA_ERR_LAUNCH;
  }
  return finish_launch(hswa::launch_decode(p, s), s);
}

}  // namespace

extern "C" {

hswa_status hswa_decode_multi(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                              const int32_t *context_lens, int32_t ns, int32_t num_queries, int32_t max_context_len,
                              void *workspace, size_t workspace_bytes, void *out, void *stream) {
  return decode_impl(layer, shape, cache, q, context_lens, ns, num_queries, max_context_len, workspace,
                     workspace_bytes, false, out, stream);
}

hswa_status hswa_decode(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                        const int32_t *context_lens, int32_t ns, int32_t max_context_len, void *workspace,
                        size_t workspace_bytes, void *out, void *stream) {
  return decode_impl(layer, shape, cache, q, context_lens, ns, 1, max_context_len, workspace, workspace_bytes, false,
                     out, stream);
}

hswa_status hswa_decode_append(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                               const void *k_new, const void *v_new, const int32_t *context_lens, int32_t ns,
                               int32_t max_context_len, void *workspace, size_t workspace_bytes, void *out,
                               void *stream) {
  return decode_impl(layer, shape, cache, q, context_lens, ns, 1, max_context_len, workspace, workspace_bytes, false,
                     out, stream, k_new, v_new, true);
}

hswa_status hswa_decode_noalloc(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache, const void *q,
                                const int32_t *context_lens, int32_t ns, int32_t max_context_len, void *out,
                                void *stream) {
  return decode_impl(layer, shape, cache, q, context_lens, ns, 1, max_context_len, nullptr, 0, true, out, stream);
}

const char *hswa_status_string(hswa_status status) {
  switch (status) {
    case HSWA_OK: return "HSWA_OK";
    case HSWA_ERR_INVALID_ARG: return "HSWA_ERR_INVALID_ARG";
    case HSWA_ERR_UNSUPPORTED: return "HSWA_ERR_UNSUPPORTED";
    case HSWA_ERR_CAPACITY: return "HSWA_ERR_CAPACITY";
    case HSWA_ERR_LAUNCH: return "HSWA_ERR_LAUNCH";
  }
  return "HSWA_UNKNOWN_STATUS";
}

}  // extern "C"
