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
// it. Each wave owns 32 rows (two 16-column MFMA groups). Per 64-key tile:
//   S^T[key][row]  = K[key][:] . Q[row][:]          (bf16 MFMA, fp32 accumulate)
//   online softmax per row in fp32 (exp2, scale*log2(e) folded in); the running
//   maximum is only raised when a score exceeds it by more than 2^8 in exp2
//   units, so the output rescale is rare (exact: numerator and denominator share
//   the stale maximum)
//   O^T[d][row]   += V^T[d][key] . P^T[key][row]    (bf16 MFMA)
// The two waves of a SIMD play ping-pong: while one runs its matrix products
// (QK^T of one tile, PV of the previous one) the other runs its softmax and
// stages tiles, and workgroup barriers swap the roles, so the matrix cores and
// the vector ALUs work at the same time.
// LDS holds the tiles in MFMA operand order (every operand read is one
// contiguous, conflict-free 1 KiB); four tile buffers let two tiles be read
// while a third is stored, and the global loads of a fourth are in flight.
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
constexpr int kBufs = 4;  // LDS tile buffers (a power of two): two being read, one stored, one loading
static_assert((kBufs & (kBufs - 1)) == 0, "buffer indices are taken modulo kBufs with a mask");
// a lane's share (16 probabilities) of a row sum above which the running
// maximum is raised
constexpr float kLaneSumLimit = 4096.f;
constexpr int kAhead = 6;  // LDS operand reads in flight ahead of the matrix products
// LDS holds each tile in MFMA operand order: every operand a wave reads (K: 16
// keys x 32 dims of a QK^T step; V^T: 16 dims x 32 keys of a PV step) is a
// contiguous 1 KiB block with lane l's 16 bytes at 16 l, so each operand read
// is one conflict-free ds_read_b128 at a per-lane base plus a constant.
//   K tile: block (h, ab, t) at ((2 h + ab) * 4 + t) KiB holds, for lane
//     r + 16 q, dims 32 t + 8 q .. +7 of tile key 32 h + 8 (r >> 2) + 4 ab + (r & 3):
//     MFMA row r of the QK^T step of half h, block ab, dim slab t. This is the
//     pool's K block layout, so an interior tile is a straight copy.
//   V^T tile: block (h, dt) at 16 KiB + (8 h + dt) KiB holds, for lane r + 16 q,
//     keys 32 h + 8 q .. +7 of dim 16 dt + r.
constexpr int kKTileBytes = kKT * kHeadDim * 2;
// Fourth word of a gfx9 buffer resource for raw (untyped) loads: 32-bit data
// format, no swizzle, no index stride.
constexpr int kBufferWord3 = 0x00020000;
constexpr int kBufBytes = 2 * kKTileBytes;

// LDS byte offset (within a buffer) of keys 32 h + 8 q .. +7 of dim d (V^T).
__device__ __forceinline__ uint32_t v_lds_off(int h, int q, int d) {
  return (uint32_t)(kKTileBytes + ((8 * h + (d >> 4)) * 64 + (d & 15) + 16 * q) * 16);
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

constexpr int kStage = kKT * kHeadDim / 8 / kThreads;  // 16-byte pieces per thread per tile (K or V)
static_assert(kStage == 2 && kKT == 64, "V staging maps piece i of a thread to 32-key block i");

// Staging maps every wave's 16-byte LDS stores onto one contiguous 1 KiB
// operand block (lane l at 16 l), so the stores are free of bank conflicts;
// thread tid (lane l of wave w) stores piece i at byte 16 tid + 8 KiB i of the
// K tile and of the V^T tile.
// V^T piece i of thread tid: dim 16 w + l % 16, keys 8 (4 i + l / 16) .. +7 of
// the tile, i.e. piece l / 16 of dim row 16 w + l % 16 of the pool's 32-key V
// block i (a wave reads one contiguous 1 KiB of the block).
// K tile pieces in pool order: piece idx (0 .. 1023) is 16-byte piece idx & 511
// of the tile's 32-key block idx >> 9 (half (idx >> 8) & 1, slab (idx >> 6) & 3,
// dim piece (idx >> 4) & 3, row idx & 15 of the block's K layout), i.e. dims
// 8 k_piece_c .. +7 of tile key k_piece_key. LDS holds it at byte 16 idx.
__device__ __forceinline__ int k_piece_key(int idx) {
  const int r = idx & 15;
  return ((idx >> 9) << 5) | ((r >> 2) << 3) | (((idx >> 8) & 1) << 2) | (r & 3);
}
__device__ __forceinline__ int k_piece_c(int idx) { return ((idx >> 6) & 3) * 4 + ((idx >> 4) & 3); }

__device__ __forceinline__ int v_piece_dim(int tid) { return 16 * (tid >> 6) + (tid & 15); }
__device__ __forceinline__ int v_piece_keys(int tid, int i) { return 4 * i + ((tid >> 4) & 3); }

struct Stage {
  u32x4 k[kStage], v[kStage];
  bool vrow;  // chunk tile: k[] holds key rows, v[] pieces follow the chunk mapping
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
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // uniform in a wave
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, hq = p.hq;
  const int shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;

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
  auto load_tile = [&](int kt, int tpage, Stage &st) __attribute__((always_inline)) {
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
  // Chunk tile: every key is one of this chunk's own (key >= P). K and V rows
  // are 256-byte runs of k_new / v_new, loaded as 16-byte pieces of a row. K
  // piece i of lane l of wave w is MFMA row l % 16 of K block (h = i,
  // ab = w / 4, slab w % 4), dims 32 (w % 4) + 8 (l / 16) .. +7, so it lands at
  // the same LDS byte as a pool piece. V piece i of lane l of wave w is key
  // 8 w + 4 i + l / 16, dims 8 (l % 16) .. +7; the store transposes those into
  // V^T (store_tile).
  auto load_tile_chunk = [&](int kt, Stage &st) __attribute__((always_inline)) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    const int r = lane & 15, ab = wave >> 2;
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int j = kt + 32 * i + 8 * (r >> 2) + 4 * ab + (r & 3);
      const bool in = j >= klo && j <= khi;
      const int c = 4 * (wave & 3) + (lane >> 4);
      const int64_t off = ((int64_t)(tok0 + (in ? j - P : 0)) * hkv + g) * kHeadDim + c * 8;
      st.k[i] = in ? ldg128(p.k_new + off) : z;
    }
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      const int j = kt + 8 * wave + 4 * i + (lane >> 4);
      const bool in = j >= klo && j <= khi;
      const int64_t off = ((int64_t)(tok0 + (in ? j - P : 0)) * hkv + g) * kHeadDim + (lane & 15) * 8;
      st.v[i] = in ? ldg128(p.v_new + off) : z;
    }
    st.vrow = true;
  };
  // Full chunk tile: every key is the chunk's own and inside [klo, khi]. The
  // tile's 64 rows of k_new / v_new start at a wave-uniform address and each
  // lane's pieces sit at fixed byte offsets from it (rows of Hkv D 2 bytes), so
  // the loads are buffer loads from a scalar resource with those offsets: no
  // per-tile vector address arithmetic and no per-lane range checks.
  const uint32_t row_bytes = (uint32_t)hkv * (kHeadDim * 2);
  const bool chunk_buf = (uint64_t)hkv * (kHeadDim * 2) * kKT <= 0x7fffffffull;
  uint32_t ch_koff[kStage], ch_voff[kStage];
  {
    const int r = lane & 15, ab = wave >> 2, c = 4 * (wave & 3) + (lane >> 4);
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      ch_koff[i] = (uint32_t)(32 * i + 8 * (r >> 2) + 4 * ab + (r & 3)) * row_bytes + (uint32_t)c * 16u;
      ch_voff[i] = (uint32_t)(8 * wave + 4 * i + (lane >> 4)) * row_bytes + (uint32_t)(lane & 15) * 16u;
    }
  }
  auto load_tile_chunk_full = [&](int kt, Stage &st) __attribute__((always_inline)) {
    const int64_t row0 = ((int64_t)(tok0 + kt - P) * hkv + g) * kHeadDim;
    const __amdgpu_buffer_rsrc_t krs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.k_new + row0), 0, kKT * row_bytes, kBufferWord3);
    const __amdgpu_buffer_rsrc_t vrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.v_new + row0), 0, kKT * row_bytes, kBufferWord3);
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      st.k[i] = __builtin_amdgcn_raw_buffer_load_b128(krs, (int)ch_koff[i], 0, 0);
      st.v[i] = __builtin_amdgcn_raw_buffer_load_b128(vrs, (int)ch_voff[i], 0, 0);
    }
    st.vrow = true;
  };
  // Interior tile: every key cached, in range and (PG >= 64) on one page whose
  // id was fetched ahead; the K tile is two 8 KiB K blocks and the V tile two
  // [D][32] blocks of 8 KiB, all contiguous: plain 16-byte loads, consecutive
  // threads at consecutive addresses.
  // The tile's two base addresses are wave-uniform (scalar registers) and each
  // load adds a fixed 32-bit per-lane byte offset (buffer loads), so a tile's
  // loads need no vector address arithmetic.
  // (The empty asm keeps the offsets opaque: the compiler would otherwise fold
  // the constant 8 KiB step between a thread's two pieces into arithmetic of
  // its own.)
  uint32_t pg_koff[kStage] = {(uint32_t)tid * 16u, (uint32_t)(tid + kThreads) * 16u};
  uint32_t pg_voff[kStage] = {(uint32_t)(v_piece_dim(tid) * 32 + ((tid >> 4) & 3) * 8) * 2u,
                              (uint32_t)(32 * kHeadDim + v_piece_dim(tid) * 32 + ((tid >> 4) & 3) * 8) * 2u};
#pragma unroll
  for (int i = 0; i < kStage; ++i) asm volatile("" : "+v"(pg_koff[i]), "+v"(pg_voff[i]));
  // For a tile on one page (PG >= 64, in-page offset a multiple of 64) both
  // pools put the page-head at the same byte offset, page * (Hkv PG D 2) +
  // g * (PG D 2), and its 32-key blocks 8 KiB apart: one scalar offset serves
  // the K and the V loads.
  const uint32_t page_bytes = (uint32_t)hkv << (shift + kHeadDimShift + 1);
  const uint64_t head_bytes = (uint64_t)g << (shift + kHeadDimShift + 1);
  auto load_tile_page = [&](int kt, int page, Stage &st) __attribute__((always_inline)) {
    const uint64_t o = (uint64_t)(uint32_t)max(page, 0) * page_bytes + head_bytes +
                       (uint64_t)(((uint32_t)kt & (uint32_t)(pg - 1)) >> 5) * 8192u;
    const char *kbase = reinterpret_cast<const char *>(pv.k_pool) + o;
    const char *vbase = reinterpret_cast<const char *>(pv.v_pool) + o;
    // buffer loads: the tile's 16 KiB from a scalar resource on its first
    // byte plus this lane's fixed 32-bit offset, so a tile's four loads need
    // no vector address arithmetic (offsets past the 16 KiB would read 0)
    const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(kbase), 0, kKTileBytes, kBufferWord3);
    const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(vbase), 0, kKTileBytes, kBufferWord3);
#pragma unroll
    for (int i = 0; i < kStage; ++i) {
      st.k[i] = __builtin_amdgcn_raw_buffer_load_b128(krs, (int)pg_koff[i], 0, 0);
      st.v[i] = __builtin_amdgcn_raw_buffer_load_b128(vrs, (int)pg_voff[i], 0, 0);
    }
    st.vrow = false;
  };
  // LDS addresses are a per-lane byte offset (fixed for the kernel) plus the
  // buffer's byte offset (a scalar), with everything else in the instruction's
  // immediate offset field.
  auto buf_off = [&](int buf) { return (uint32_t)__builtin_amdgcn_readfirstlane(buf * kBufBytes); };
  auto lds128 = [&](uint32_t off) { return reinterpret_cast<u32x4 *>(s_lds + off); };
  // LDS offsets of this thread's pieces: piece 1 is 8 KiB after piece 0, except
  // for the V^T pieces of a chunk tile, dims 8 (l % 16) + 2 m and + 1
  // (m = l / 16) of keys 8 w .. +7, which are 16 bytes apart.
  const uint32_t st_k0 = tid * 16;
  const uint32_t st_v0 = kKTileBytes + tid * 16;
  const uint32_t st_vrow0 = v_lds_off(wave >> 2, wave & 3, 8 * (lane & 15) + 2 * (lane >> 4));
  // 4 x 4 transpose of dwords across the lanes l, l ^ 16, l ^ 32, l ^ 48: the
  // lane in 16-lane row m enters with dword j of its row m in t[j] and leaves
  // with dword m of rows 0..3 in w[0..3] (a swap with l ^ 32, then with l ^ 16).
  auto transpose4 = [&](const u32x4 &t, uint32_t (&w)[4]) {
    const auto a = __builtin_amdgcn_permlane32_swap(t[0], t[2], false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(t[1], t[3], false, false);
    const auto c = __builtin_amdgcn_permlane16_swap((uint32_t)a[0], (uint32_t)b[0], false, false);
    const auto d = __builtin_amdgcn_permlane16_swap((uint32_t)a[1], (uint32_t)b[1], false, false);
    w[0] = (uint32_t)c[0];
    w[1] = (uint32_t)c[1];
    w[2] = (uint32_t)d[0];
    w[3] = (uint32_t)d[1];
  };
  auto store_tile = [&](int buf, Stage &st) __attribute__((always_inline)) {
    static_assert(kStage == 2, "two pieces per thread");
    const uint32_t bo = buf_off(buf);
    *lds128(bo + st_k0) = st.k[0];
    *lds128(bo + st_k0 + kKTileBytes / 2) = st.k[1];
    if (st.vrow) {
      // The lanes l % 16 + 16 m (m = 0..3) of a wave hold an 8 x 8 block: keys
      // 8 w + 4 i + m (piece i) x dims 8 (l % 16) .. +7. After the transposes
      // lane m holds dims 2 m, 2 m + 1 of keys 8 w .. +7 (w[k]); byte permutes
      // split them into one V^T piece per dim, which replace the pieces in
      // place (so both kinds of tile store the same registers and the stores
      // need no copies).
      uint32_t w[8];
      transpose4(st.v[0], *reinterpret_cast<uint32_t(*)[4]>(&w[0]));
      transpose4(st.v[1], *reinterpret_cast<uint32_t(*)[4]>(&w[4]));
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        st.v[0][j] = __builtin_amdgcn_perm(w[2 * j + 1], w[2 * j], 0x05040100u);
        st.v[1][j] = __builtin_amdgcn_perm(w[2 * j + 1], w[2 * j], 0x07060302u);
      }
    }
    // V^T pieces: a pool tile's two pieces sit 8 KiB apart at st_v0, a chunk
    // tile's 16 bytes apart at st_vrow0
    const uint32_t va = bo + (st.vrow ? st_vrow0 : st_v0);
    *lds128(va) = st.v[0];
    *lds128(va + (uint32_t)__builtin_amdgcn_readfirstlane(st.vrow ? 16 : kKTileBytes / 2)) = st.v[1];
  };

  float m[kCG], lsum[kCG];  // m: running maximum in exp2 units
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
  auto fetch = [&](int kt, int page, Stage &st) __attribute__((always_inline)) {
    if (page >= 0 && interior(kt)) load_tile_page(kt, page, st);
    else if (kt >= P && chunk_buf && kt >= klo && kt + kKT - 1 <= khi) load_tile_chunk_full(kt, st);
    else if (kt >= P) load_tile_chunk(kt, st);
    else load_tile(kt, page, st);
  };

  // QK^T of one half tile: S^T for keys kt + 32h .. +31.
  const uint32_t op_lane = lane * 16;
  auto qk_half = [&](int buf, int h, f32x4 (&sc)[2][kCG]) {
    const uint32_t a = buf_off(buf) + op_lane + h * (kKTileBytes / 2);
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      sc[0][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
      sc[1][cg] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 ka = *lds128(a + 1024 * t);
      const u32x4 kb = *lds128(a + 4096 + 1024 * t);
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
    // kt laundered: the per-lane bounds below are then formed here, in the
    // masked tiles only, not carried through the loop as vector induction
    // variables that every tile would update
    int ktl = kt;
    asm volatile("" : "+s"(ktl));
    const int j0 = ktl + 32 * h + 8 * q;
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
  // Lazy raise of the running maximum, checked after the fact. The
  // exponentials of a tile are taken against the running maximum m as it
  // stands, and each lane adds up its 16 probabilities of a column (its share
  // of the row sum). Only if some lane's share exceeds 2^12 (a ballot; an
  // infinite sum counts) is the exact column maximum formed across the 4 lanes
  // that share a column, m raised to it, the output and the row sum rescaled,
  // and the tile's exponentials taken again. Otherwise every probability is
  // below 2^12 and m stays: the result is the same either way, because
  // numerator and denominator share m, and the 2^12 bound keeps both far
  // inside the fp32 and bf16 ranges. The running maximum is kept in exp2
  // units (score * scale * log2 e) and starts at -FLT_MAX, a finite value
  // whatever the scale: exp2 of a masked score (-inf) is then 0 with no NaN
  // from (-inf) - (-inf), and the first finite score always raises it (its
  // probability overflows to infinity; alpha = exp2(-huge) = 0).
  // The exponentials give the bf16 P^T operands; the row sums use the same
  // bf16-rounded probabilities as the PV product.
  auto tile_exp = [&](f32x4 (&sc)[2][2][kCG], u32x4 (&pf)[2][kCG], float (&ts)[kCG]) {
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) {
      const float mc = m[cg];
      ts[cg] = 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float pr[8];
#pragma unroll
        for (int ab = 0; ab < 2; ++ab)
#pragma unroll
          for (int i = 0; i < 4; ++i) pr[4 * ab + i] = fast_exp2(fmaf(sc[h][ab][cg][i], c2, -mc));
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) pf[h][cg][jj] = pack_bf16x2(pr[2 * jj], pr[2 * jj + 1]);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) ts[cg] = dot2_bf16_ones(pf[h][cg][jj], ts[cg]);
      }
    }
  };
  auto softmax_tile = [&](f32x4 (&sc)[2][2][kCG], u32x4 (&pf)[2][kCG]) {
    float ts[kCG];
    tile_exp(sc, pf, ts);
    bool raise = false;
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) raise = raise || !(ts[cg] <= kLaneSumLimit);
    if (__builtin_amdgcn_ballot_w64(raise) != 0) {
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) {
        const float a8[8] = {sc[0][0][cg][0], sc[0][0][cg][1], sc[0][0][cg][2], sc[0][0][cg][3],
                             sc[0][1][cg][0], sc[0][1][cg][1], sc[0][1][cg][2], sc[0][1][cg][3]};
        const float b8[8] = {sc[1][0][cg][0], sc[1][0][cg][1], sc[1][0][cg][2], sc[1][0][cg][3],
                             sc[1][1][cg][0], sc[1][1][cg][1], sc[1][1][cg][2], sc[1][1][cg][3]};
        const float cmax = max_xor32(max_xor16(max2(max8(a8), max8(b8)))) * c2;
        const bool up = cmax > m[cg];
        const float alpha = up ? fast_exp2(m[cg] - cmax) : 1.f;
        m[cg] = up ? cmax : m[cg];
        lsum[cg] *= alpha;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) acc[cg][dt] *= alpha;
      }
      tile_exp(sc, pf, ts);
    }
#pragma unroll
    for (int cg = 0; cg < kCG; ++cg) lsum[cg] += ts[cg];
  };
  // O^T += V^T P^T for one half tile.
  auto load_v = [&](int buf, int h, u32x4 (&vf)[8]) {
    const uint32_t a = buf_off(buf) + kKTileBytes + op_lane + h * (kKTileBytes / 2);  // keys 32h + 8q .. +7
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) vf[dt] = *lds128(a + 1024 * dt);
  };
  auto pv_ops = [&](const u32x4 (&vf)[8], const u32x4 (&pf)[kCG]) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int cg = 0; cg < kCG; ++cg) acc[cg][dt] = mfma16x16x32(vf[dt], pf[cg], acc[cg][dt]);
  };

  // ---- tile loop ----
  // The waves form two groups, A (waves 0-3) and B (waves 4-7), one wave of
  // each on every SIMD. A tile is processed in two phases: a matrix phase
  // (QK^T of tile j and PV of tile j-1, both on MFMA with operands from LDS)
  // and a softmax phase (VALU: mask, exponentials, row sums, plus this
  // thread's share of the tile staging: LDS stores, global loads, address
  // arithmetic). Group B runs its phases offset from group A's (see the loop),
  // so that on every SIMD one wave's matrix products overlap the other wave's
  // softmax, and the two matrix phases overlap in part. Each thread stores its
  // share of a tile two (group A) or one (group B) barrier intervals before
  // the tile is first read; the global loads of a tile go out one tile before
  // its store.
  auto pv_tile = [&](int buf, const u32x4 (&pf)[2][kCG]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      u32x4 vf[8];
      load_v(buf, h, vf);
      pv_ops(vf, pf[h]);
    }
  };

  Stage st;
  fetch(kt0, tile_page(kt0), st);
  store_tile(0, st);
  if (ntiles > 1) {
    fetch(kt0 + kKT, tile_page(kt0 + kKT), st);
    store_tile(1, st);
  }
  if (ntiles > 2) fetch(kt0 + 2 * kKT, tile_page(kt0 + 2 * kKT), st);
  __syncthreads();
  const bool lag = wave >= kThreads / kWave / 2;  // group B

  f32x4 sc[2][2][kCG];
  u32x4 pf[2][kCG];
  // matrix phase: PV of tile jt-1, QK^T of tile jt, at raised issue priority
  // so that the other wave's softmax takes the issue slots the matrix
  // products leave free
  auto matrix_phase = [&](int jt) __attribute__((always_inline)) {
    const int buf = jt & (kBufs - 1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(2);
    if (jt > 0) {
      pv_tile((jt + kBufs - 1) & (kBufs - 1), pf);
      // operand reads run kAhead reads ahead of the products that use them
      __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
      for (int i = 0; i < 16 - kAhead; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * kAhead, 0);
    }
    qk_half(buf, 0, sc[0]);
    qk_half(buf, 1, sc[1]);
    __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 1);
#pragma unroll
    for (int i = 0; i < 16 - kAhead; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * kAhead, 1);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_setprio(0);
  };
  // softmax phase of tile jt, with this thread's share of the staging: tile
  // jt+2 from registers to LDS, tile jt+3's global loads
  auto softmax_phase = [&](int jt) __attribute__((always_inline)) {
    const int kt = kt0 + jt * kKT;
    if (jt + 2 < ntiles) store_tile((jt + 2) & (kBufs - 1), st);
    if (jt + 3 < ntiles) fetch(kt + 3 * kKT, tile_page(kt + 3 * kKT), st);
    if (needs_mask(kt)) {
      mask_half(kt, 0, sc[0]);
      mask_half(kt, 1, sc[1]);
    }
    softmax_tile(sc, pf);
  };
  // One barrier per tile. Between barriers t and t+1 group A runs the matrix
  // phase of tile t, then its softmax phase; group B first the softmax phase
  // of tile t-1, then the matrix phase of tile t. A wave of B thus starts its
  // matrix products while its SIMD partner is still in its own, and the
  // partner's softmax runs under the rest of them. Between those barriers the
  // tiles read are t (K) and t-1 (V); the stores go to tile t+2 (group A) and
  // t+1 (group B), whose buffers were last read (as tiles t-2 and t-3) before
  // barrier t, and a stored tile is first read after a further barrier.
  auto tile_barrier = [&]() {
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
  };
  if (!lag) {
    for (int jt = 0; jt < ntiles; ++jt) {
      matrix_phase(jt);
      softmax_phase(jt);
      tile_barrier();
    }
  } else {
    matrix_phase(0);
    tile_barrier();
    for (int jt = 1; jt < ntiles; ++jt) {
      softmax_phase(jt - 1);
      matrix_phase(jt);
      tile_barrier();
    }
    softmax_phase(ntiles - 1);
  }
  pv_tile((ntiles + kBufs - 1) & (kBufs - 1), pf);

  // ---- normalise and write ----
#pragma unroll
  for (int cg = 0; cg < kCG; ++cg) {
    const float l = sum_xor32(sum_xor16(lsum[cg]));
    const float inv = 1.f / l;
    const int row = wave * (16 * kCG) + cg * 16 + r;
    const int po = row / G, head = row - po * G;
    uint16_t *orow = p.out + ((int64_t)(tok0 + q0 + (cval[cg] ? po : 0)) * hq + (int64_t)g * G + head) * kHeadDim;
    u32x2 w[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      w[dt][0] = pack_bf16x2(acc[cg][dt][0] * inv, acc[cg][dt][1] * inv);
      w[dt][1] = pack_bf16x2(acc[cg][dt][2] * inv, acc[cg][dt][3] * inv);
    }
    store_out_row(orow, w, q, cval[cg]);
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillParams &p, hipStream_t stream) {
  if (p.ns <= 0 || p.max_chunk_len <= 0 || p.total_tokens <= 0) return hipSuccess;
  if (p.pool.window > 0 && prefill_run_fits(p)) return launch_prefill_run(p, stream);
  if (p.pool.window > 0 && p.pool.window <= kPrefillWindowMax) return launch_prefill_window(p, stream);
  const int npos = kRows / p.group;
  const int64_t ntq = (p.max_chunk_len + npos - 1) / npos;
  const int64_t pairs_per_xcd = ((int64_t)p.ns * p.hkv + kXcds - 1) / kXcds;
  const int64_t grid = pairs_per_xcd * ntq * kXcds;
  return launch_kernel(prefill_kernel, dim3((unsigned)grid), dim3(kThreads), stream, p);
}

}  // namespace hswa
