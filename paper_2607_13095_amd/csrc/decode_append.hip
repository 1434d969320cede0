// Decode step of one new token per sequence with its append fused in.
//
// "KVCache Storage Analysis": an SWA layer's decode reads only the window,
// a few tens of KiB per (sequence, KV head), so its time is the latency of a
// short chain of dependent loads rather than HBM bandwidth; a model with many
// SWA layers pays that chain, and a launch, for each of them. This kernel
// stores the step's new K / V row in its slot and decodes the step's query in
// one launch: the new key enters the attention straight from the input
// registers, so the decode never waits for the store.
//
// One workgroup per (sequence, KV head, group of up to 16 query heads); one
// wave per 32-key chunk of the range (the window of an SWA layer, the whole
// context of a short FULL layer), so that every chunk's loads are in flight at
// once; the waves combine their softmax states through LDS. The range's table
// lookups are made as early as possible: an SWA ring row (at most 64 entries)
// is read by the lanes of every wave at the start, next to the query and the
// context length, and chunk pages then come from a lane read.
// Per chunk, as in the decode kernel: S^T = K . Q^T and O^T += V^T . P^T on the
// bf16 matrix cores with the GQA heads as the 16 columns, online softmax in
// fp32 with exp2, running maximum in exp2 units raised lazily.
#include <cfloat>

#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kAChunk = 32;
constexpr int kACols = 16;
constexpr int kAMaxWaves = 8;
constexpr float kARescaleLog2 = 8.f;

__device__ __forceinline__ u32x4 ldnt128_global(const void *p) {
  return __builtin_nontemporal_load((global_u32x4 *)p);
}

// LDS of the combine: per wave its 8 accumulator vectors of every lane, then
// its 16 column maxima and sums.
constexpr int kAStateBytes = 8 * kWave * 16 + 2 * kACols * 4;

__global__ __launch_bounds__(kWave * kAMaxWaves) void decode_append_kernel(DecodeParams p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char s_state[];
  const PoolView &pv = p.pool;
  const int nw = (int)(blockDim.x / kWave);
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int r = lane & 15, q = lane >> 4;
  const int hkv = p.hkv, shift = pv.pg_shift, pg = 1 << shift;
  const float c2 = p.scale_log2;
  const int hchunks = (p.group + kACols - 1) / kACols;
  const int item = (int)blockIdx.x;
  const int b = item / (hkv * hchunks);
  const int gy = item - b * hkv * hchunks;
  const int g = gy / hchunks, hc = gy - g * hchunks;
  const int col = hc * kACols + r;
  const bool colv = col < p.group;
  const int64_t row = (int64_t)b * p.hq + (int64_t)g * p.group + (colv ? col : 0);
  const int64_t kvrow = ((int64_t)b * hkv + g) * kHeadDim;  // the new token's K / V row

  // Independent loads first (all unconditional, so that the waits on them stay
  // exact): the ring's table row (lane i: entry min(i, R - 1); entry 0 without
  // a ring), the query, the new K / V pieces this lane stores if it is the
  // writer, the context length.
  const bool lane_ring = pv.ring > 0 && pv.ring <= kWave;
  const int tabv = pv.table[(int64_t)b * pv.stride + min(lane, max(pv.ring, 1) - 1)];
  u32x4 qf[4];
  {
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 v = ldg128(p.q + row * kHeadDim + 32 * t + 8 * q);
      qf[t] = colv ? v : z;
    }
  }
  const u32x4 kapp = ldg128(p.k_new + kvrow + 8 * r);
  const uint16_t vapp0 = p.v_new[kvrow + lane], vapp1 = p.v_new[kvrow + lane + 64];
  const int ring_page = lane < pv.ring && tabv >= 0 && tabv < pv.num_pages ? tabv : -1;
  const int ctx = min(p.ctx_lens[b], p.max_ctx);
  if (ctx < 1) {  // no token: nothing stored, a zero output row
    if (wid == 0 && colv) {
      const u32x2 z = {0u, 0u};
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) *reinterpret_cast<u32x2 *>(p.out + row * kHeadDim + 16 * dt + 4 * q) = z;
    }
    return;
  }
  const int pos = ctx - 1;
  const int kb = pv.window > 0 ? max(0, pos - pv.window + 1) : 0;
  const int cfirst = kb & ~(kAChunk - 1);
  const int nchunks = ((pos - cfirst) >> 5) + 1;
  // physical page of logical page lp (-1: not a valid page)
  auto page_of = [&](int lp) {
    if (lane_ring) return __builtin_amdgcn_readlane(ring_page, lp % pv.ring);
    const int e = pv.ring > 0 ? lp % pv.ring : lp;
    const int v = pv.table[(int64_t)b * pv.stride + e];  // e < stride: checked on the host
    return (v >= 0 && v < pv.num_pages) ? v : -1;
  };

  const int app_page = page_of(pos >> shift);

  // Lane offsets inside one 32-key chunk (PG >= 32: a chunk lies in one page):
  // K half a (keys 8 i + j, j < 4, at MFMA row 4 i + j), half b 4 KiB on; the
  // V^T block of dims 16 dt + r, keys 8 q .. +7.
  const uint32_t koff = lane * 16;
  const uint32_t voff = (r * 32 + 8 * q) * 2;
  const int key_a = 8 * (r >> 2) + (r & 3);  // this lane's K row key in half a (+4 in half b)

  float m = -FLT_MAX, lsum = 0.f;
  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c = wid; c < nchunks; c += nw) {
    const int cbase = cfirst + c * kAChunk;
    const int page = page_of(cbase >> shift);
    const int64_t pg64 = max(page, 0);
    const char *kbase = reinterpret_cast<const char *>(pv.k_pool) +
                        ((((pg64 * hkv + g) << shift) + (cbase & (pg - 1))) * kHeadDim) * 2;
    const char *vbase = reinterpret_cast<const char *>(pv.v_pool) +
                        ((((pg64 * hkv + g) << shift) << kHeadDimShift) +
                         ((int64_t)((cbase & (pg - 1)) >> 5) << (5 + kHeadDimShift))) * 2;
    // the new key (offset o of the last chunk; -1 elsewhere) comes from k_new / v_new
    const int o = pos - cbase < kAChunk ? pos - cbase : -1;
    const char *knew = reinterpret_cast<const char *>(p.k_new + kvrow + 8 * q);
    u32x4 ka[4], kbv[4], v[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      ka[t] = ldnt128_global(key_a == o ? knew + 64 * t : kbase + koff + 1024 * t);
      kbv[t] = ldnt128_global(key_a + 4 == o ? knew + 64 * t : kbase + koff + 4096 + 1024 * t);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) v[dt] = ldnt128_global(vbase + voff + dt * 1024);
    uint32_t vn[8];
    if (o >= 0) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) vn[dt] = p.v_new[kvrow + 16 * dt + r];
    }

    // S^T[key][head]: rows of half a then half b
    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = sa;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      sa = mfma16x16x32(ka[t], qf[t], sa);
      sb = mfma16x16x32(kbv[t], qf[t], sb);
    }
    // lane holds keys cbase + 8 q .. +7 of column r
    const uint32_t keep = page >= 0 ? key_range_bits(cbase + 8 * q, kb, pos) : 0u;
    float s[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i] = sa[i];
      s[4 + i] = sb[i];
    }
    if (__builtin_amdgcn_ballot_w64(keep != 0xFFu) != 0) {
#pragma unroll
      for (int i = 0; i < 8; ++i) s[i] = (keep >> i) & 1u ? s[i] : -INFINITY;
    }
    const float lmax = max8(s) * c2;
    if (__builtin_amdgcn_ballot_w64(lmax > m + kARescaleLog2) != 0) {
      const float cmax = max_xor32(max_xor16(lmax));
      const bool up = cmax > m + kARescaleLog2;
      const float alpha = up ? fast_exp2(m - cmax) : 1.f;
      m = up ? cmax : m;
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[dt] *= alpha;
    }
    float pr[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pr[i] = fast_exp2(fmaf(s[i], c2, -m));
    u32x4 pf;
#pragma unroll
    for (int j = 0; j < 4; ++j) pf[j] = pack_bf16x2(pr[2 * j], pr[2 * j + 1]);
#pragma unroll
    for (int j = 0; j < 4; ++j) lsum = dot2_bf16_ones(pf[j], lsum);

    // V^T: the new key's value replaces its slot's element; keys outside the
    // range are zeroed (their slots may hold anything, NaN included)
    if (o >= 0 && (o >> 3) == q) {
      const int w = (o & 7) >> 1, sh = 16 * (o & 1);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) v[dt][w] = (v[dt][w] & ~(0xFFFFu << sh)) | (vn[dt] << sh);
    }
    if (keep != 0xFFu) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) v[dt] = keep_bf16x8(v[dt], keep);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[dt] = mfma16x16x32(v[dt], pf, acc[dt]);
  }

  // The append: wave 0 of the first head group stores the new row in its slot
  // (no wave of the launch reads that slot: the new key came from the input).
  if (hc == 0 && wid == 0 && app_page >= 0) {
    const int o = pos & (pg - 1);
    if (lane < 16) stg128(pv.k_pool + k_offset(pv, app_page, hkv, g, o, 8 * lane), kapp);
    pv.v_pool[v_offset(pv, app_page, hkv, g, o, lane)] = vapp0;
    pv.v_pool[v_offset(pv, app_page, hkv, g, o, lane + 64)] = vapp1;
  }

  // Combine the waves' states; wave slice s (s < 4, taken by waves s, s + nw, ...)
  // normalises and writes dims 32 s .. 32 s + 31 of every column.
  f32x4 *s_o = reinterpret_cast<f32x4 *>(s_state);                       // [nw][8][64]
  float *s_m = reinterpret_cast<float *>(s_state + nw * 8 * kWave * 16);  // [nw][16]
  float *s_l = s_m + nw * kACols;                                         // [nw][16]
  {
    const float l = sum_xor32(sum_xor16(lsum));
    if (q == 0) {
      s_m[wid * kACols + r] = m;
      s_l[wid * kACols + r] = l;
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) s_o[(wid * 8 + dt) * kWave + lane] = acc[dt];
  }
  __syncthreads();
  if (!colv) return;
  float mx = -FLT_MAX;
  for (int w = 0; w < nw; ++w) mx = fmaxf(mx, s_m[w * kACols + r]);
  float l = 0.f;
  for (int w = 0; w < nw; ++w) l += fast_exp2(s_m[w * kACols + r] - mx) * s_l[w * kACols + r];
  const float inv = l > 0.f ? 1.f / l : 0.f;
  for (int sl = wid; sl < 4; sl += nw) {
    // this lane's 8 output dims d0 .. d0 + 7: dims 16 dt + 4 q' + i of the
    // accumulators with dt = 2 sl + q / 2 and q' = 2 (q % 2), 2 (q % 2) + 1
    const int d0 = 32 * sl + 8 * q;
    const int sdt = 2 * sl + (q >> 1), sln = r + 32 * (q & 1);
    f32x4 o0 = {0.f, 0.f, 0.f, 0.f}, o1 = o0;
    for (int w = 0; w < nw; ++w) {
      const float wgt = fast_exp2(s_m[w * kACols + r] - mx);
      o0 += wgt * s_o[(w * 8 + sdt) * kWave + sln];
      o1 += wgt * s_o[(w * 8 + sdt) * kWave + sln + 16];
    }
    u32x4 wv;
    wv[0] = pack_bf16x2(o0[0] * inv, o0[1] * inv);
    wv[1] = pack_bf16x2(o0[2] * inv, o0[3] * inv);
    wv[2] = pack_bf16x2(o1[0] * inv, o1[1] * inv);
    wv[3] = pack_bf16x2(o1[2] * inv, o1[3] * inv);
    *reinterpret_cast<u32x4 *>(p.out + row * kHeadDim + d0) = wv;
  }
}

}  // namespace

// Chunks a whole-range item may span: the window (W keys touch at most
// ceil((W - 1) / 32) + 1 aligned chunks), at most the context's.
static int range_chunks(const DecodeParams &p) {
  const int ctx_chunks = (p.max_ctx + kAChunk - 1) / kAChunk;
  return p.pool.window > 0 ? min(ctx_chunks, (p.pool.window + kAChunk - 2) / kAChunk + 1) : ctx_chunks;
}

bool decode_append_fused(const DecodeParams &p) {
  return p.nq == 1 && p.max_splits == 1 && p.pool.pg_shift >= 5 && range_chunks(p) <= kAMaxWaves;
}

hipError_t launch_decode_append(const DecodeParams &p, hipStream_t stream) {
  if (p.ns <= 0) return hipSuccess;
  const int nw = max(1, range_chunks(p));
  const int hchunks = (p.group + kACols - 1) / kACols;
  const int64_t items = (int64_t)p.ns * p.hkv * hchunks;
  void *args[] = {const_cast<DecodeParams *>(&p)};
  return hipLaunchKernel(reinterpret_cast<const void *>(decode_append_kernel), dim3((unsigned)items),
                         dim3(kWave * nw), args, (size_t)nw * kAStateBytes, stream);
}

}  // namespace hswa
