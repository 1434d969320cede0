// Chunked prefill attention over a cached prefix.
//
// "Compute Analysis": chunked prefill is largely compute-bound, and an SWA
// layer only needs the keys inside its window, so tiles outside the window are
// never visited. Keys below the prefix length P come from the paged cache (FULL:
// the block table; SWA: the ring), keys from P on come from the chunk's own
// k_new / v_new (the chunk is appended to the cache only after this kernel).
//
// Work unit: one workgroup (8 waves, two per SIMD) per (tile of 256 query rows,
// KV head, sequence). A query row is a (position, query head) pair of the KV
// head's GQA group, so one K/V tile in LDS serves every query head that shares
// it. Each wave owns 32 rows (two 16-column MFMA groups); two waves per SIMD
// let one wave's softmax run while the other's matrix products do. Per 64-key
// tile:
//   S^T[key][row]  = K[key][:] . Q[row][:]          (bf16 MFMA, fp32 accumulate)
//   online softmax per row in fp32 (exp2, scale*log2(e) folded in); the running
//   maximum is only raised when a score exceeds it by more than 2^8 in exp2
//   units, so the output rescale is rare (exact: numerator and denominator share
//   the stale maximum)
//   O^T[d][row]   += V^T[d][key] . P^T[key][row]    (bf16 MFMA)
// K is staged in LDS as rows (in the order the MFMA rows consume them), V as its
// transpose, both with padded rows so that the 16 lanes reading one operand hit
// distinct banks; four LDS tile buffers let tile j+3 be stored while tiles j and
// j+1 are read, and the global loads of tile j+4 are in flight meanwhile.
// Keys outside the workgroup's range are staged as zeros, so NaN or stale data
// in unused cache slots never reaches an accumulator; per-element masks are
// applied only on tiles that cross the causal diagonal, the window edge or the
// range ends. Workgroups are mapped so that each XCD works through the query
// tiles of a few (sequence, KV head) pairs at a time and shares their K/V in L2.
#include <cfloat>
#include <type_traits>

#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kThreads = 512;
constexpr int kRows = 256;  // query rows per workgroup
constexpr int kKT = 64;     // keys per tile
constexpr int kCG = 2;      // 16-column MFMA groups per wave
constexpr int kXcds = 8;
constexpr int kBufs = 4;  // LDS tile buffers: two being read, one written, one spare
constexpr float kRescaleLog2 = 8.f;
// LDS rows are padded by 16 bytes, so the 16 lanes that read one MFMA operand
// (16 consecutive LDS rows at one column) spread over all banks, and every
// address of a wave's operand reads is a per-lane base plus a constant.
constexpr int kKRow = kHeadDim + 8;  // K tile row (one key), in bf16 elements
constexpr int kVRow = kKT + 8;       // V^T tile row (one dim), in bf16 elements

// LDS row of key k (0..63) of a tile: the MFMA row that consumes it. Within each
// 32-key half, keys 8a+c (c < 4) feed row 4a+c of block a (rows 0..15) and keys
// 8a+4+c feed row 4a+c of block b (rows 16..31).
__device__ __forceinline__ int k_lds_row(int k) {
  return (k & 32) | ((k & 4) << 2) | ((k >> 3 & 3) << 2) | (k & 3);
}

__device__ __forceinline__ int64_t prefix_page(const PoolView &pv, int b, int key, bool &ok) {
  int lp = key >> pv.pg_shift;
  if (pv.ring > 0) lp %= pv.ring;
  if (lp >= pv.stride) {
    ok = false;
    return 0;
  }
  const int64_t page = pv.table[(int64_t)b * pv.stride + lp];
  ok = page >= 0 && page < pv.num_pages;
  return ok ? page : 0;
}

constexpr int kKTileBytes = kKT * kKRow * 2;
constexpr int kBufBytes = kKTileBytes + kHeadDim * kVRow * 2;
constexpr int kStage = kKT * kHeadDim / 8 / kThreads;  // 16-byte pieces per thread per tile (K or V)
static_assert(kStage == 2 && kKT == 64, "V staging maps piece i of a thread to 32-key block i");

// V^T tile staging: piece i of thread tid holds dim tid / 4 and keys
// 8 * (4 i + tid % 4) .. +7 of the tile, which in the pool is the 16 bytes at
// element 8 * tid of the tile's 32-key block i.
// K tile pieces in pool order: piece idx (0 .. 1023) is 16-byte piece idx & 511
// of the tile's 32-key block idx >> 9 (half (idx >> 8) & 1, slab (idx >> 6) & 3,
// dim piece (idx >> 4) & 3, row idx & 15 of the block's K layout), i.e. dims
// 8 k_piece_c .. +7 of tile key k_piece_key, which LDS holds in row k_piece_row.
__device__ __forceinline__ int k_piece_key(int idx) {
  const int r = idx & 15;
  return ((idx >> 9) << 5) | ((r >> 2) << 3) | (((idx >> 8) & 1) << 2) | (r & 3);
}
__device__ __forceinline__ int k_piece_c(int idx) { return ((idx >> 6) & 3) * 4 + ((idx >> 4) & 3); }
__device__ __forceinline__ int k_piece_row(int idx) { return ((idx >> 8) << 4) | (idx & 15); }

__device__ __forceinline__ int v_piece_dim(int tid) { return tid >> 2; }
__device__ __forceinline__ int v_piece_keys(int tid, int i) { return 4 * i + (tid & 3); }

struct Stage {
  u32x4 k[kStage], v[kStage];
  bool vrow;  // v[] holds 8 dims of one key (as k[]) instead of 8 keys of one dim
};

__global__ __launch_bounds__(kThreads) void prefill_kernel(PrefillParams p) {
  // kBufs tile buffers, each a K tile then a V^T tile (byte offsets below)
  __shared__ __attribute__((aligned(16))) unsigned char s_lds[kBufs * kBufBytes];

  const PoolView &pv = p.pool;
  const int G = p.group;
  const int npos = kRows / G;  // positions per workgroup

  // XCD-aware order. Workgroup ids are dealt to the XCDs round-robin; the
  // (sequence, KV head) pairs are dealt the same way, pair x + 8k to XCD x, so
  // every query tile of a pair runs on one XCD and shares its K/V in that L2,
  // while pairs of unequal length (different prefixes) spread over all XCDs.
  // Within a pair the longest query tiles (the last ones) go first.
  const int ntq = (p.max_chunk_len + npos - 1) / npos;
  const int npairs = p.ns * p.hkv;
  const int xcd = (int)(blockIdx.x % kXcds);
  const int local = (int)(blockIdx.x / kXcds);
  const int k = local / ntq;
  const int tq = ntq - 1 - (local - k * ntq);
  const int pair = xcd + kXcds * k;
  if (pair >= npairs) return;
  const int b = pair / p.hkv, g = pair - b * p.hkv;

  const int tok0 = p.cu_seqlens[b];
  // never step outside q / k_new / v_new / out, whatever the device offsets say
  const int C = min(min(p.cu_seqlens[b + 1], p.total_tokens) - tok0, p.max_chunk_len);
  const int P = p.prefix_lens[b];
  const int q0 = tq * npos;
  if (q0 >= C || P < 0 || tok0 < 0) return;
  const int q1 = min(C, q0 + npos) - 1;
  const int pfirst = P + q0, plast = P + q1;
  const int W = pv.window;
  const int klo = W > 0 ? max(0, pfirst - W + 1) : 0;
  const int khi = plast;

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, hq = p.hq;
  const int shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;
  const float thresh = kRescaleLog2 / c2;  // in raw score units

  // Q^T operands and the position of each of this lane's columns.
  u32x4 qf[kCG][4];
  int cpos[kCG], clo[kCG];
  bool cval[kCG];
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) {
    const int row = wave * (16 * kCG) + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    cval[cg] = q0 + po <= q1;
    cpos[cg] = P + q0 + po;
    clo[cg] = W > 0 ? max(0, cpos[cg] - W + 1) : 0;
    const int64_t tok = tok0 + q0 + (cval[cg] ? po : 0);
    const uint16_t *qrow = p.q + (tok * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 v = ldg128(qrow + 32 * t + 8 * q);
      const u32x4 z = {0u, 0u, 0u, 0u};
      qf[cg][t] = cval[cg] ? v : z;
    }
  }

  // ---- staging: global -> registers -> LDS ----
  const bool page_tiles = shift >= 6;  // PG >= 64: a 64-key tile lies on one page
  // General tile (range ends, the prefix / chunk boundary, PG < 64): per-key
  // source and range checks. With PG >= 64 the tile's page (tpage, from the
  // lane table) serves every cached key; otherwise each key looks its page up.
  auto cached_page = [&](int j, int tpage, bool &ok) -> int64_t {
    if (page_tiles) {
      ok = tpage >= 0;
      return ok ? tpage : 0;
    }
    return prefix_page(pv, b, j, ok);
  };
  auto load_tile = [&](int kt, int tpage, Stage &st) {
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int idx = tid + kThreads * i;
      const int c = k_piece_c(idx);
      const int j = kt + k_piece_key(idx);
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j >= klo && j <= khi) {
        if (j < P) {
          bool ok;
          const int64_t page = cached_page(j, tpage, ok);
          if (ok) v = ldg128(pv.k_pool + k_offset(pv, page, hkv, g, j & (pg - 1), c * 8));
        } else {
          v = ldg128(p.k_new + ((int64_t)(tok0 + j - P) * hkv + g) * kHeadDim + c * 8);
        }
      }
      st.k[i] = v;
    }
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int d = v_piece_dim(tid), kc = v_piece_keys(tid, i);
      const int j0 = kt + 8 * kc;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (j0 >= klo && j0 + 7 <= khi && j0 + 7 < P) {
        bool ok;
        const int64_t page = cached_page(j0, tpage, ok);
        if (ok) v = ldg128(pv.v_pool + v_offset(pv, page, hkv, g, j0 & (pg - 1), d));
      } else if (j0 + 7 >= klo && j0 <= khi) {
        uint32_t e[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int j = j0 + t;
          e[t] = 0u;
          if (j >= klo && j <= khi) {
            if (j < P) {
              bool ok;
              const int64_t page = cached_page(j, tpage, ok);
              if (ok) e[t] = pv.v_pool[v_offset(pv, page, hkv, g, j & (pg - 1), d)];
            } else {
              e[t] = p.v_new[((int64_t)(tok0 + j - P) * hkv + g) * kHeadDim + d];
            }
          }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = e[2 * t] | (e[2 * t + 1] << 16);
      }
      st.v[i] = v;
    }
    st.vrow = false;
  };
  // Chunk tile: every key is one of this chunk's own (key >= P), so its K and
  // V rows are 256-byte runs of k_new / v_new: both are loaded as 16-byte
  // pieces of a key's row, and V is transposed on its way into LDS.
  auto load_tile_chunk = [&](int kt, Stage &st) {
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int idx = tid + kThreads * i;
      const int j = kt + (idx >> 4);
      const bool in = j >= klo && j <= khi;
      const int64_t off = ((int64_t)(tok0 + (in ? j - P : 0)) * hkv + g) * kHeadDim + (idx & 15) * 8;
      const u32x4 z = {0u, 0u, 0u, 0u};
      st.k[i] = in ? ldg128(p.k_new + off) : z;
      st.v[i] = in ? ldg128(p.v_new + off) : z;
    }
    st.vrow = true;
  };
  // Interior tile: every key cached, in range and (PG >= 64) on one page whose
  // id was fetched ahead; the K tile is two 8 KiB K blocks and the V tile two
  // [D][32] blocks of 8 KiB, all contiguous: plain 16-byte loads, consecutive
  // threads at consecutive addresses.
  auto load_tile_page = [&](int kt, int page, Stage &st) {
    const int64_t pg64 = max(page, 0);
    const int off = kt & (pg - 1);
    const uint16_t *kbase = pv.k_pool + k_offset(pv, pg64, hkv, g, off, 0);
    const uint16_t *vbase = pv.v_pool + v_offset(pv, pg64, hkv, g, off, 0);
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int idx = tid + kThreads * i;
      st.k[i] = ldg128(kbase + idx * 8);
      st.v[i] = ldg128(vbase + i * (32 * kHeadDim) + tid * 8);
    }
    st.vrow = false;
  };
  // LDS addresses are a per-lane byte offset (fixed for the kernel) plus the
  // buffer's byte offset (a scalar), with everything else in the instruction's
  // immediate offset field.
  auto buf_off = [&](int buf) { return (uint32_t)__builtin_amdgcn_readfirstlane(buf * kBufBytes); };
  auto lds128 = [&](uint32_t off) { return reinterpret_cast<u32x4 *>(s_lds + off); };
  // K piece 0 of this thread in pool order (cached tiles) or row order (chunk
  // tiles); piece 1 is 32 rows on in both.
  const uint32_t st_k0 = (k_piece_row(tid) * kKRow + k_piece_c(tid) * 8) * 2;
  const uint32_t st_k0_row = (k_lds_row(tid >> 4) * kKRow + (tid & 15) * 8) * 2;
  const uint32_t st_v0 = kKTileBytes + (v_piece_dim(tid) * kVRow + v_piece_keys(tid, 0) * 8) * 2;
  const uint32_t st_vrow0 = kKTileBytes + ((tid & 15) * 8 * kVRow + (tid >> 4)) * 2;  // row form, piece 0
  auto store_tile = [&](int buf, const Stage &st) {
    static_assert(kStage == 2, "two pieces per thread");
    const uint32_t bo = buf_off(buf);
    // piece 1 of K is key + 32 (LDS row + 32), of V keys + 32 (block 1)
    const uint32_t k0 = st.vrow ? st_k0_row : st_k0;
    *lds128(bo + k0) = st.k[0];
    *lds128(bo + k0 + 32 * kKRow * 2) = st.k[1];
    if (!st.vrow) {
      *lds128(bo + st_v0) = st.v[0];
      *lds128(bo + st_v0 + 32 * 2) = st.v[1];
    } else {
      // dims 8c .. 8c+7 of key tid/16 (+32 for piece 1): one 2-byte store per dim
#pragma unroll
      for (int i = 0; i < kStage; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          *reinterpret_cast<uint16_t *>(s_lds + bo + st_vrow0 + (e * kVRow + 32 * i) * 2) =
              (uint16_t)(st.v[i][e >> 1] >> (16 * (e & 1)));
    }
  };

  float m[kCG], lsum[kCG];
  f32x4 acc[kCG][8];
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) {
    m[cg] = -FLT_MAX;
    lsum[cg] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[cg][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // One 64-key tile, processed as two 32-key halves (QK^T, softmax, PV each),
  // which keeps the score and probability registers of a wave at 32 + 16.
  // ---- pipelined tile loop ----
  // Work is split into half tiles of 32 keys. The QK^T of the next half is
  // issued before the softmax of the current one, so the matrix cores and the
  // VALU work of a wave can overlap; LDS holds three tiles (the two being read
  // and the one being written), with one barrier per tile.
  const int kt0 = klo & ~(kKT - 1);
  const int ntiles = (khi - kt0) / kKT + 1;
  // A tile is "interior" when all of its keys are cached, inside [klo, khi]
  // and (PG >= 64) on a single page; its page id is looked up one tile ahead.
  auto interior = [&](int kt) { return page_tiles && kt >= klo && kt + kKT - 1 <= khi && kt + kKT - 1 < P; };
  // Page ids of interior tiles come from a per-wave window of the block table:
  // lane i holds the physical page of logical page tab_lp0 + i, refilled every
  // 64 pages, and a tile's id is read with v_readlane (no per-tile memory
  // round trip). -1 marks a tile that is not interior or whose page is invalid.
  int tab_page = -1, tab_lp0 = -(1 << 30);
  // For PG >= 64 every 64-key tile lies on one logical page: its physical page
  // comes from the lane table for any tile that starts in the cached prefix
  // (-1 for a chunk tile or a page that is not valid).
  auto tile_page = [&](int kt) {
    if (!page_tiles || kt >= P) return -1;
    const int lp = kt >> shift;
    if (lp - tab_lp0 >= kWave || lp < tab_lp0) {
      tab_lp0 = lp;
      const int lpl = lp + lane;
      int page = -1;
      if (lpl <= ((P - 1) >> shift)) {
        const int e = pv.ring > 0 ? lpl % pv.ring : lpl;
        if (e < pv.stride) {
          const int64_t v = pv.table[(int64_t)b * pv.stride + e];
          page = (v >= 0 && v < pv.num_pages) ? (int)v : -1;
        }
      }
      tab_page = page;
    }
    return __builtin_amdgcn_readlane(tab_page, lp - tab_lp0);
  };
  auto fetch = [&](int kt, int page, Stage &st) {
    if (page >= 0 && interior(kt)) load_tile_page(kt, page, st);
    else if (kt >= P) load_tile_chunk(kt, st);
    else load_tile(kt, page, st);
  };

  // QK^T of one half tile: S^T for keys kt + 32h .. +31.
  const uint32_t qk_lane = (r * kKRow + 8 * q) * 2;
  const uint32_t pv_lane = kKTileBytes + (r * kVRow + 8 * q) * 2;
  auto qk_half = [&](int buf, int h, f32x4 (&sc)[2][kCG]) {
    // MFMA row r of block a is LDS row 32h + r, of block b row 32h + 16 + r
    const uint32_t a = buf_off(buf) + qk_lane + 32 * h * kKRow * 2;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      sc[0][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
      sc[1][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 ka = *lds128(a + 64 * t);
      const u32x4 kb = *lds128(a + 16 * kKRow * 2 + 64 * t);
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) {
        sc[0][cg] = mfma16x16x32(ka, qf[cg][t], sc[0][cg]);
        sc[1][cg] = mfma16x16x32(kb, qf[cg][t], sc[1][cg]);
      }
    }
  };
  // Per-element mask of a half tile on the diagonal, window edge or range ends.
  auto mask_half = [&](int kt, int h, f32x4 (&sc)[2][kCG]) {
    // this lane's 8 keys are kt + 32h + 8q + e, e = 4 ab + i; allowed e form
    // the interval [lo_e, hi_e] of the column's visible keys
    const int j0 = kt + 32 * h + 8 * q;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      const int lo_e = max(max(clo[cg], klo) - j0, 0);
      const int hi_e = min(min(cpos[cg], khi) - j0, 7);
      const uint32_t bits = hi_e < lo_e ? 0u : ((2u << hi_e) - 1u) & ~((1u << lo_e) - 1u);
#pragma unroll
      for (int ab = 0; ab < 2; ++ab)
#pragma unroll
        for (int i = 0; i < 4; ++i) sc[ab][cg][i] = (bits >> (4 * ab + i)) & 1u ? sc[ab][cg][i] : -INFINITY;
    }
  };
  auto needs_mask = [&](int kt) {
    return kt + kKT - 1 > pfirst || kt < klo || kt + kKT - 1 > khi || (W > 0 && kt < plast - W + 1);
  };
  // Lazy raise of the running maximum. Each lane compares the maximum of its
  // own 8 scores with m + thresh; only if some lane exceeds it (a ballot) is
  // the exact column maximum formed across the 4 lanes that share a column
  // and the output rescaled. Otherwise every probability stays below 2^8.
  // The running maximum starts at -FLT_MAX, a finite value: exp2 of a masked
  // score (-inf) is then 0 with no NaN from (-inf) - (-inf), and the first
  // finite score always raises it (alpha = exp2(-huge) = 0).
  auto softmax_max = [&](f32x4 (&sc)[2][kCG]) {
    float lmax[kCG];
    bool raise = false;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      const float v8[8] = {sc[0][cg][0], sc[0][cg][1], sc[0][cg][2], sc[0][cg][3],
                           sc[1][cg][0], sc[1][cg][1], sc[1][cg][2], sc[1][cg][3]};
      lmax[cg] = max8(v8);
      raise = raise || lmax[cg] > m[cg] + thresh;
    }
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) {
        const float cmax = max_xor32(max_xor16(lmax[cg]));
        const bool up = cmax > m[cg] + thresh;
        const float alpha = up ? fast_exp2((m[cg] - cmax) * c2) : 1.f;
        m[cg] = up ? cmax : m[cg];
        lsum[cg] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[cg][dt] *= alpha;
      }
    }
  };
  // exp2 and the bf16 P^T operand; the row sums use the same bf16-rounded
  // probabilities as the PV product.
  auto softmax_exp = [&](f32x4 (&sc)[2][kCG], u32x4 (&pf)[kCG]) {
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      const float mc = m[cg] * c2;
      float pr[8];
#pragma unroll
      for (int ab = 0; ab < 2; ++ab)
#pragma unroll
        for (int i = 0; i < 4; ++i) pr[4 * ab + i] = fast_exp2(fmaf(sc[ab][cg][i], c2, -mc));
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) pf[cg][jj] = pack_bf16x2(pr[2 * jj], pr[2 * jj + 1]);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) lsum[cg] = dot2_bf16_ones(pf[cg][jj], lsum[cg]);
    }
  };
  // O^T += V^T P^T for one half tile.
  auto load_v = [&](int buf, int h, u32x4 (&vf)[8]) {
    const uint32_t a = buf_off(buf) + pv_lane + 64 * h;  // keys 32h + 8q .. +7
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) vf[dt] = *lds128(a + 16 * dt * kVRow * 2);
  };
  auto pv_ops = [&](const u32x4 (&vf)[8], const u32x4 (&pf)[kCG]) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) acc[cg][dt] = mfma16x16x32(vf[dt], pf[cg], acc[cg][dt]);
  };

  // Prologue: tiles 0..2 in LDS, tile 3's loads in flight, QK^T of (0, 0).
  Stage st;
  fetch(kt0, tile_page(kt0), st);
  store_tile(0, st);
  if (ntiles > 1) {
    fetch(kt0 + kKT, tile_page(kt0 + kKT), st);
    store_tile(1, st);
  }
  if (ntiles > 2) {
    fetch(kt0 + 2 * kKT, tile_page(kt0 + 2 * kKT), st);
    store_tile(2, st);
  }
  if (ntiles > 3) fetch(kt0 + 3 * kKT, tile_page(kt0 + 3 * kKT), st);
  __syncthreads();
  f32x4 s_a[2][kCG], s_b[2][kCG];
  qk_half(0, 0, s_a);

  for (int jt = 0; jt < ntiles; ++jt) {
    const int kt = kt0 + jt * kKT;
    const int buf = jt % kBufs;
    const bool masked = needs_mask(kt);
    u32x4 pf[kCG], vf[8];
    // softmax of (jt, 0) with the QK^T of (jt, 1) issued alongside, PV of (jt, 0)
    load_v(buf, 0, vf);
    if (masked) mask_half(kt, 0, s_a);
    softmax_max(s_a);
    qk_half(buf, 1, s_b);
    softmax_exp(s_a, pf);
    pv_ops(vf, pf);
    // Every wave is past its last read of tile jt-1: tile jt+3 (in registers
    // since the previous iteration) overwrites its buffer, and tile jt+4's
    // loads go out, a whole iteration ahead of their store.
    __syncthreads();
    if (jt + 3 < ntiles) store_tile((jt + 3) % kBufs, st);
    if (jt + 4 < ntiles) fetch(kt + 4 * kKT, tile_page(kt + 4 * kKT), st);
    // softmax of (jt, 1) with the QK^T of (jt + 1, 0) issued alongside (it is
    // unconditional so that it interleaves with the exponentials; after the
    // last tile it reads a stale buffer and the result is never used), PV of
    // (jt, 1)
    load_v(buf, 1, vf);
    if (masked) mask_half(kt, 1, s_b);
    softmax_max(s_b);
    qk_half((jt + 1) % kBufs, 0, s_a);
    softmax_exp(s_b, pf);
    pv_ops(vf, pf);
  }

  // ---- normalise and write ----
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) {
    const float l = sum_xor32(sum_xor16(lsum[cg]));
    if (!cval[cg]) continue;
    const float inv = 1.f / l;
    const int row = wave * (16 * kCG) + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    uint16_t *orow = p.out + ((int64_t)(tok0 + q0 + po) * hq + (int64_t)g * G + head) * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      u32x2 w;
      w[0] = pack_bf16x2(acc[cg][dt][0] * inv, acc[cg][dt][1] * inv);
      w[1] = pack_bf16x2(acc[cg][dt][2] * inv, acc[cg][dt][3] * inv);
      *reinterpret_cast<u32x2 *>(orow + 16 * dt + 4 * q) = w;
    }
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillParams &p, hipStream_t stream) {
  if (p.ns <= 0 || p.max_chunk_len <= 0 || p.total_tokens <= 0) return hipSuccess;
  const int npos = kRows / p.group;
  const int64_t ntq = (p.max_chunk_len + npos - 1) / npos;
  const int64_t pairs_per_xcd = ((int64_t)p.ns * p.hkv + kXcds - 1) / kXcds;
  const int64_t grid = pairs_per_xcd * ntq * kXcds;
  return launch_kernel(prefill_kernel, dim3((unsigned)grid), dim3(kThreads), stream, p);
}

}  // namespace hswa
