// Internal launcher interface between the C ABI layer (api.hip) and the
// kernels. Arguments are validated by the caller before these are reached.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hswa {

constexpr int kHeadDim = 128;  // the only head dim the kernels are built for
constexpr int kHeadDimShift = 7;
// Both pools store a page-head as PG / B blocks of B = min(PG, 32) consecutive
// keys. V blocks are transposed ([D][B]): the V^T operand of a 32-key chunk of
// one head is one contiguous 8 KiB run. K blocks hold two halves (keys whose
// in-block offset has bit 2 clear, then set), each as four 32-dim slabs of
// [B/2 keys][32 dims] with the 16-byte pieces in bf16-MFMA lane order: the 16
// keys x 32 dims of one QK^T operand are one contiguous 1 KiB run (B = 32).
constexpr int kVBlockShiftMax = 5;

// Pool geometry and block table of one layer, as the kernels see it.
struct PoolView {
  uint16_t *k_pool;       // bf16 [num_pages][Hkv][PG/B][2][D/32][4][B/2][8]
  uint16_t *v_pool;       // bf16 [num_pages][Hkv][PG/B][D][B]
  int64_t num_pages;
  const int32_t *table;   // int32 [ns][stride]
  int32_t stride;
  int32_t pg_shift;       // log2(page size)
  int32_t vb_shift;       // log2(B) = min(pg_shift, 5), the key block of both pools
  int32_t ring;           // ring pages R (SWA) or 0 (FULL)
  int32_t window;         // SWA window W, or 0 for FULL
};

struct AppendParams {
  PoolView pool;
  const uint16_t *k_new;  // [T][Hkv][D]
  const uint16_t *v_new;  // [T][Hkv][D]
  const int32_t *cu_seqlens;
  const int32_t *start_pos;
  int64_t *slot_out;      // [T] or null
  int32_t ns, total_tokens, hkv;
  // Decode-step mode (ctx_lens non-null): token b is sequence b's, at position
  // min(ctx_lens[b], max_ctx) - 1 (none if that is negative); cu_seqlens and
  // start_pos are not read.
  const int32_t *ctx_lens;
  int32_t max_ctx;
};

struct DecodeParams {
  PoolView pool;
  const uint16_t *q;      // [ns][Hq][D]
  const int32_t *ctx_lens;
  uint16_t *out;          // [ns][Hq][D]
  float *ws_o;            // FULL split partials [ns * nq * Hq][max_splits][D]
  float *ws_lse;          // [ns * nq * Hq][max_splits]
  int32_t ns, hq, hkv, group, max_ctx;
  int32_t nq;             // queries per sequence, at positions ctx - nq .. ctx - 1 (q, out: [ns][nq][Hq][D])
  int32_t split_len;      // FULL split: fewest keys of a wave's span (a multiple of 32)
  int32_t max_splits;     // pieces a (row) may have; 1 => single pass, no workspace
  int32_t span_waves;     // FULL split: waves the chunk order is divided over (set at launch)
  int32_t item_cols;      // (query, head) columns of one item (set at launch)
  float scale_log2;       // scale * log2(e)
  const uint16_t *k_new;  // decode step: the new token's K / V rows [ns][Hkv][D]
  const uint16_t *v_new;
  // FULL split decode of one new token per sequence, PG >= 32: the kernel also
  // stores the token (k_new / v_new) in its slot and takes its key from them
  int32_t split_append;
};

struct PrefillParams {
  PoolView pool;
  const uint16_t *q;      // [T][Hq][D]
  const uint16_t *k_new;  // [T][Hkv][D]
  const uint16_t *v_new;  // [T][Hkv][D]
  const int32_t *cu_seqlens;
  const int32_t *prefix_lens;
  uint16_t *out;          // [T][Hq][D]
  int32_t ns, total_tokens, max_chunk_len, hq, hkv, group;
  float scale_log2;
};

hipError_t launch_kv_append(const AppendParams &p, hipStream_t stream);
hipError_t launch_decode(const DecodeParams &p, hipStream_t stream);
// Decode step with its append in the same launch (decode_append.hip): one
// query per sequence, whole-range items of at most 8 chunks, PG >= 32.
bool decode_append_fused(const DecodeParams &p);
hipError_t launch_decode_append(const DecodeParams &p, hipStream_t stream);
hipError_t launch_prefill(const PrefillParams &p, hipStream_t stream);
// SWA prefill whose window is at most kPrefillWindowMax keys: 128 query rows
// per workgroup over the window's keys only (prefill_window.hip).
constexpr int kPrefillWindowMax = 512;
hipError_t launch_prefill_window(const PrefillParams &p, hipStream_t stream);
// SWA prefill with a GQA group of at least 8 and W + 256 / G - 1 <= 160: one
// workgroup per run of position tiles, the window's chunks in an LDS ring
// (prefill_run.hip).
bool prefill_run_fits(const PrefillParams &p);
hipError_t launch_prefill_run(const PrefillParams &p, hipStream_t stream);

// Device address of the library's fixed scratch array on the current device
// (looked up once per device).
hipError_t noalloc_scratch(void **ptr);

// Fewest keys of a FULL decode wave's span; a multiple of 256.
int32_t decode_split_len(int32_t ns, int32_t hkv, int32_t group, int32_t max_ctx);

}  // namespace hswa
