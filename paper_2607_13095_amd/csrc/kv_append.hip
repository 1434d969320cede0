// KV append: slot mapping and scatter of new K/V rows into the paged pools.
//
// Dual-pool layout ("KVCache Dual-Pool Design"): a FULL layer keeps every
// position; an SWA layer keeps a ring of R = ceil(W/PG)+1 pages per sequence,
// and the ring overwrite is the out-of-window eviction that follows every chunk
// and every decode step ("SWA-Aware Prefix Cache Tree").
//
// One workgroup handles 8 consecutive tokens of the flattened batch for one KV
// head. A token's K row goes to the pool as sixteen 16-byte pieces (the K
// blocks are stored in MFMA-operand slabs); V pages are stored as transposed
// blocks of B = min(PG, 32) keys ([D][B] per block and head), so 8 tokens that
// land on 8 consecutive, 8-aligned slots of one page are written as one 16-byte
// store per dim; anything else falls back to 2-byte stores.
#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kTokPerBlock = 8;
constexpr int kThreads = 256;
constexpr int kLdsSeqs = 4096;  // batches up to this size search cu_seqlens in LDS

// Sequence of flattened token t: the b with cu[b] <= t < cu[b+1] (-1 if none).
// `cu` is the LDS copy of cu_seqlens when it fits, else the global array.
__device__ int find_seq(const int32_t *cu, int ns, int t) {
  int lo = 0, hi = ns;  // answer in [0, ns)
  if (ns <= 0 || t < cu[0] || t >= cu[ns]) return -1;
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (cu[mid] <= t) lo = mid; else hi = mid;
  }
  return lo;
}

__device__ int64_t slot_of_token(const AppendParams &p, const int32_t *cu, int t) {
  int b;
  int64_t j, len_after;
  if (p.ctx_lens) {  // decode step: token t is sequence t's
    b = t;
    len_after = min(p.ctx_lens[b], p.max_ctx);
    j = len_after - 1;
  } else {
    b = find_seq(cu, p.ns, t);
    if (b < 0) return -1;
    const int64_t start = p.start_pos[b];
    j = start + (t - cu[b]);
    len_after = start + (cu[b + 1] - cu[b]);
  }
  if (j < 0) return -1;
  const PoolView &pv = p.pool;
  const int64_t pg = int64_t(1) << pv.pg_shift;
  int64_t lp = j >> pv.pg_shift;
  if (pv.ring > 0) {
    if (j < len_after - pv.ring * pg) return -1;  // the ring keeps the latest R*PG
    lp = lp % pv.ring;
  }
  if (lp >= pv.stride) return -1;
  const int64_t page = pv.table[int64_t(b) * pv.stride + lp];
  if (page < 0 || page >= pv.num_pages) return -1;
  return page * pg + (j & (pg - 1));
}

// Grid: (groups of 8 tokens, KV heads). Each workgroup moves 8 tokens of one
// KV head: 8 K rows of 256 bytes and 8 x 128 V values.
__global__ __launch_bounds__(kThreads) void kv_append_kernel(AppendParams p) {
  __shared__ int64_t s_slot[kTokPerBlock];
  __shared__ int32_t s_cu[kLdsSeqs + 1];
  const int t0 = blockIdx.x * kTokPerBlock;
  const int g = blockIdx.y;
  const int tid = threadIdx.x;
  const int ntok = min(kTokPerBlock, p.total_tokens - t0);
  // One coalesced load of cu_seqlens instead of a chain of dependent loads in
  // the binary search.
  const bool lds_cu = p.ns <= kLdsSeqs && !p.ctx_lens;
  if (lds_cu) {
    for (int i = tid; i <= p.ns; i += kThreads) s_cu[i] = p.cu_seqlens[i];
  }
  __syncthreads();
  if (tid < ntok) {
    const int64_t s = slot_of_token(p, lds_cu ? s_cu : p.cu_seqlens, t0 + tid);
    s_slot[tid] = s;
    if (p.slot_out && g == 0) p.slot_out[t0 + tid] = s;
  }
  __syncthreads();

  const PoolView &pv = p.pool;
  const int pg = 1 << pv.pg_shift;
  const int hkv = p.hkv;
  constexpr int kRow16 = kHeadDim / 8;  // 16-byte pieces per K row

  // K rows: threads 0..127 copy the 16-byte pieces of 8 rows.
  if (tid < kTokPerBlock * kRow16) {
    const int tok = tid / kRow16, c = tid % kRow16;
    const int64_t s = tok < ntok ? s_slot[tok] : -1;
    if (s >= 0) {
      const int64_t page = s >> pv.pg_shift, off = s & (pg - 1);
      const u32x4 v = ldg128(p.k_new + ((int64_t)(t0 + tok) * hkv + g) * kHeadDim + c * 8);
      stg128(pv.k_pool + k_offset(pv, page, hkv, g, (int)off, c * 8), v);
    }
  }

  // V: transposed pages.
  bool run = ntok == kTokPerBlock && s_slot[0] >= 0 && (s_slot[0] & 7) == 0;
#pragma unroll
  for (int i = 1; i < kTokPerBlock; ++i) run = run && s_slot[i] == s_slot[0] + i;
  if (run) {
    // 8 consecutive, 8-aligned slots of one page: one 16-byte store per dim
    if (tid < kHeadDim) {
      const int d = tid;
      const int64_t page = s_slot[0] >> pv.pg_shift, off = s_slot[0] & (pg - 1);
      const uint16_t *src = p.v_new + ((int64_t)t0 * hkv + g) * kHeadDim + d;
      u32x4 w;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint32_t lo = src[(int64_t)(2 * k) * hkv * kHeadDim];
        const uint32_t hi = src[(int64_t)(2 * k + 1) * hkv * kHeadDim];
        w[k] = lo | (hi << 16);
      }
      stg128(pv.v_pool + v_offset(pv, page, hkv, g, (int)off, d), w);
    }
  } else {
    for (int i = tid; i < ntok * kHeadDim; i += kThreads) {
      const int tok = i / kHeadDim, d = i - tok * kHeadDim;
      const int64_t s = s_slot[tok];
      if (s < 0) continue;
      const int64_t page = s >> pv.pg_shift, off = s & (pg - 1);
      pv.v_pool[v_offset(pv, page, hkv, g, (int)off, d)] = p.v_new[((int64_t)(t0 + tok) * hkv + g) * kHeadDim + d];
    }
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendParams &p, hipStream_t stream) {
  if (p.total_tokens <= 0) return hipSuccess;
  const int blocks = (p.total_tokens + kTokPerBlock - 1) / kTokPerBlock;
  return launch_kernel(kv_append_kernel, dim3(blocks, p.hkv), dim3(kThreads), stream, p);
}

}  // namespace hswa
