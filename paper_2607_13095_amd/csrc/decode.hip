// Decode attention over the paged KV cache (one query per sequence).
//
// "KVCache Storage Analysis": decode is memory-bound, its cost follows the KV
// bytes read; SWA layers read at most W keys from the per-sequence ring, FULL
// layers read the whole context.
//
// Work unit: one workgroup (4 waves) per (key range, KV head, sequence, group of
// up to 16 query heads of that KV head). Every wave walks 32-key chunks of the
// range and runs both products on the bf16 matrix cores with the GQA query
// heads as the 16 MFMA columns:
//   S^T[key][head]  = K[key][:] . Q[head][:]        (K rows straight from HBM)
//   O^T[d][head]   += V^T[d][key] . P^T[key][head]   (V pages are stored [D][PG])
// The 32 keys of a chunk are assigned to MFMA rows so that the score tile comes
// out with each lane holding 8 consecutive keys of one head, which is exactly
// the lane layout the PV product needs for P^T: no shuffle between the two.
// Softmax is online per chunk in fp32 (exp2 with scale*log2(e) folded in).
// The 4 waves are merged through LDS at the end. A FULL layer whose context is
// split into several pieces writes fp32 (o, log2-sum-exp) partials that a second
// kernel merges; an SWA layer (or a single piece) writes bf16 output directly.
#include "hswa_common.h"
#include "hswa_launch.h"

namespace hswa {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kChunk = 32;
constexpr int kCols = 16;        // query heads per workgroup (MFMA columns)
constexpr int kORow = kHeadDim + 4;

__device__ __forceinline__ int64_t lookup_page(const PoolView &pv, int b, int key, bool &ok) {
  int lp = key >> pv.pg_shift;
  if (pv.ring > 0) lp %= pv.ring;
  const int64_t page = pv.table[(int64_t)b * pv.stride + lp];
  ok = page >= 0 && page < pv.num_pages;
  return ok ? page : 0;
}

template <bool kSplit>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeParams p) {
  __shared__ float s_m[kWaves][kCols];
  __shared__ float s_l[kWaves][kCols];
  __shared__ __attribute__((aligned(16))) float s_o[kWaves][kCols][kORow];

  const PoolView &pv = p.pool;
  const int split = blockIdx.x;
  const int hchunks = (p.group + kCols - 1) / kCols;
  const int g = blockIdx.y / hchunks;
  const int hc = blockIdx.y - g * hchunks;
  const int b = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int r = lane & 15, q = lane >> 4;
  const int nheads = min(kCols, p.group - hc * kCols);
  const int head0 = g * p.group + hc * kCols;
  const int hkv = p.hkv;
  const int shift = pv.pg_shift;
  const int pg = 1 << shift;

  const int ctx = min(p.ctx_lens[b], p.max_ctx);
  if (ctx < 1) {
    if (!kSplit) {
      for (int i = tid; i < nheads * (kHeadDim / 2); i += kThreads) {
        const int h = i / (kHeadDim / 2), dp = i - h * (kHeadDim / 2);
        reinterpret_cast<uint32_t *>(p.out + ((int64_t)b * p.hq + head0 + h) * kHeadDim)[dp] = 0u;
      }
    }
    return;
  }
  const int pos = ctx - 1;
  int kb, ke;
  if (kSplit) {
    kb = split * p.split_len;
    if (kb > pos) return;
    ke = min(pos, kb + p.split_len - 1);
  } else {
    kb = pv.window > 0 ? max(0, pos - pv.window + 1) : 0;
    ke = pos;
  }

  // Q^T operand: lane holds head r, dims 32t + 8q .. +7 for step t.
  u32x4 qf[4];
  {
    const bool hv = r < nheads;
    const uint16_t *qrow = p.q + ((int64_t)b * p.hq + head0 + (hv ? r : 0)) * kHeadDim;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const u32x4 v = ldg128(qrow + 32 * t + 8 * q);
      const u32x4 z = {0u, 0u, 0u, 0u};
      qf[t] = hv ? v : z;
    }
  }

  const float c2 = p.scale_log2;
  const int cfirst = kb & ~(kChunk - 1);
  const int nchunks = ((ke - cfirst) >> 5) + 1;
  const int klo8 = kb & ~7, khi8 = ke & ~7;

  float m = -INFINITY, lsum = 0.f;
  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c = wave; c < nchunks; c += kWaves) {
    const int cbase = cfirst + c * kChunk;
    // K rows of this lane: keys cbase + 8*(r/4) + (r%4) (+4 for the second tile)
    const int ka = min(max(cbase + 8 * (r >> 2) + (r & 3), kb), ke);
    const int kb2 = min(max(cbase + 8 * (r >> 2) + 4 + (r & 3), kb), ke);
    const int kv0 = cbase + 8 * q;                  // the 8 keys whose scores / V this lane holds
    const int kvg = min(max(kv0, klo8), khi8);
    bool oka, okb, okv;
    const int64_t pa = lookup_page(pv, b, ka, oka);
    const int64_t pb = lookup_page(pv, b, kb2, okb);
    const int64_t pvv = lookup_page(pv, b, kvg, okv);

    const uint16_t *krow_a = pv.k_pool + (((pa * hkv + g) << shift) + (ka & (pg - 1))) * kHeadDim;
    const uint16_t *krow_b = pv.k_pool + (((pb * hkv + g) << shift) + (kb2 & (pg - 1))) * kHeadDim;
    const uint16_t *vcol = pv.v_pool + ((pvv * hkv + g) * kHeadDim << shift) + (kvg & (pg - 1));

    u32x4 kfa[4], kfb[4], vf[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      kfa[t] = ldg128(krow_a + 32 * t + 8 * q);
      kfb[t] = ldg128(krow_b + 32 * t + 8 * q);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) vf[dt] = ldg128(vcol + ((int64_t)(16 * dt + r) << shift));

    f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      sa = mfma16x16x32(kfa[t], qf[t], sa);
      sb = mfma16x16x32(kfb[t], qf[t], sb);
    }

    uint32_t keep = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) keep |= (uint32_t)(kv0 + i >= kb && kv0 + i <= ke) << i;
    if (!okv) keep = 0;

    float s[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i] = (keep >> i) & 1u ? sa[i] : -INFINITY;
      s[4 + i] = (keep >> (4 + i)) & 1u ? sb[i] : -INFINITY;
    }
    float cmax = s[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) cmax = fmaxf(cmax, s[i]);
    cmax = wave_max_xor(cmax, 16);
    cmax = wave_max_xor(cmax, 32);
    const float mnew = fmaxf(m, cmax);
    const float mc = mnew == -INFINITY ? 0.f : mnew * c2;
    const float alpha = fast_exp2(m * c2 - mc);
    float pr[8], psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      pr[i] = fast_exp2(fmaf(s[i], c2, -mc));
      psum += pr[i];
    }
    lsum = lsum * alpha + psum;
    m = mnew;

    u32x4 pf;
#pragma unroll
    for (int j = 0; j < 4; ++j) pf[j] = pack_bf16x2(pr[2 * j], pr[2 * j + 1]);
    if (keep != 0xFFu) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) vf[dt] = keep_bf16x8(vf[dt], keep);
    }
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      acc[dt] *= alpha;
      acc[dt] = mfma16x16x32(vf[dt], pf, acc[dt]);
    }
  }

  // Merge the 4 waves.
  lsum = wave_sum_xor(lsum, 16);
  lsum = wave_sum_xor(lsum, 32);
  if (q == 0) {
    s_m[wave][r] = m;
    s_l[wave][r] = lsum;
  }
  __syncthreads();
  float mall = s_m[0][r];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) mall = fmaxf(mall, s_m[w][r]);
  const float f = m == -INFINITY ? 0.f : fast_exp2((m - mall) * c2);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) {
    f32x4 v = acc[dt] * f;
    *reinterpret_cast<f32x4 *>(&s_o[wave][r][16 * dt + 4 * q]) = v;
  }
  __syncthreads();

  // Thread -> (head h, dims 2*(tid%16) + 32*k).
  const int h = tid >> 4;
  if (h >= nheads) return;
  float mh = s_m[0][h];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) mh = fmaxf(mh, s_m[w][h]);
  float fw[kWaves], ltot = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    fw[w] = s_m[w][h] == -INFINITY ? 0.f : fast_exp2((s_m[w][h] - mh) * c2);
    ltot += fw[w] * s_l[w][h];
  }
  const float inv = 1.f / ltot;
  const int64_t row = (int64_t)b * p.hq + head0 + h;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int d = 2 * (tid & 15) + 32 * k;
    float o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      o0 += s_o[w][h][d];
      o1 += s_o[w][h][d + 1];
    }
    o0 *= inv;
    o1 *= inv;
    if (kSplit) {
      float *dst = p.ws_o + (row * p.max_splits + split) * kHeadDim + d;
      dst[0] = o0;
      dst[1] = o1;
    } else {
      reinterpret_cast<uint32_t *>(p.out + row * kHeadDim)[d >> 1] = pack_bf16x2(o0, o1);
    }
  }
  if (kSplit && (tid & 15) == 0) p.ws_lse[row * p.max_splits + split] = mh * c2 + __log2f(ltot);
}

// Log-sum-exp merge of the split partials: one wave per (sequence, query head).
__global__ __launch_bounds__(kThreads) void decode_merge_kernel(DecodeParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t idx = (int64_t)blockIdx.x * kWaves + (threadIdx.x / kWave);
  if (idx >= (int64_t)p.ns * p.hq) return;
  const int b = (int)(idx / p.hq);
  const int ctx = min(p.ctx_lens[b], p.max_ctx);
  uint32_t *dst = reinterpret_cast<uint32_t *>(p.out + idx * kHeadDim) + lane;
  if (ctx < 1) {
    *dst = 0u;
    return;
  }
  const int nsplit = (ctx - 1) / p.split_len + 1;
  const float *lse = p.ws_lse + idx * p.max_splits;
  float mx = -INFINITY;
  for (int s = 0; s < nsplit; ++s) mx = fmaxf(mx, lse[s]);
  float wsum = 0.f, o0 = 0.f, o1 = 0.f;
  const float *po = p.ws_o + idx * p.max_splits * kHeadDim + 2 * lane;
  for (int s = 0; s < nsplit; ++s) {
    const float w = fast_exp2(lse[s] - mx);
    wsum += w;
    o0 = fmaf(w, po[(int64_t)s * kHeadDim], o0);
    o1 = fmaf(w, po[(int64_t)s * kHeadDim + 1], o1);
  }
  const float inv = 1.f / wsum;
  *dst = pack_bf16x2(o0 * inv, o1 * inv);
}

}  // namespace

int32_t decode_split_len(int32_t ns, int32_t hkv, int32_t group, int32_t max_ctx) {
  const int64_t units = (int64_t)ns * hkv * ((group + kCols - 1) / kCols);
  int32_t len = 1024;
  while (len > 256 && units * ((max_ctx + len - 1) / len) < 2048) len /= 2;
  // keep the number of pieces bounded for very long contexts
  const int64_t min_len = ((int64_t)max_ctx + 255) / 256;
  while (len < min_len) len *= 2;
  return len;
}

hipError_t launch_decode(const DecodeParams &p, hipStream_t stream) {
  if (p.ns <= 0) return hipSuccess;
  const int hchunks = (p.group + kCols - 1) / kCols;
  const dim3 grid(p.max_splits, p.hkv * hchunks, p.ns);
  if (p.max_splits > 1) {
    hipLaunchKernelGGL(decode_kernel<true>, grid, dim3(kThreads), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t rows = (int64_t)p.ns * p.hq;
    hipLaunchKernelGGL(decode_merge_kernel, dim3((unsigned)((rows + kWaves - 1) / kWaves)), dim3(kThreads), 0,
                       stream, p);
  } else {
    hipLaunchKernelGGL(decode_kernel<false>, grid, dim3(kThreads), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace hswa
