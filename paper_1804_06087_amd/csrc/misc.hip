// Memory-bound kernels of the hot path: input staging, pooling, spatial reductions,
// embedding gather, concatenation, the fp32 direct convolution, and the ensemble
// combine (softmax per model, mean over the selected models, first-index argmax) and
// the majority-vote combine.
#include "kernels.h"

namespace rafiki {

LaunchEvents& launch_events() {
  static thread_local LaunchEvents ev;
  return ev;
}

__device__ __forceinline__ float bf2f(uint32_t b16) { return __uint_as_float(b16 << 16); }
__device__ __forceinline__ uint32_t f2bf(float f) {   // nearest, ties to even (finite)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// 8 consecutive channels as floats, from bf16 or fp32 storage.
__device__ __forceinline__ void load8(const void* p, long long off, int bf16, float v[8]) {
  if (bf16) {
    const uint4 q = *(const uint4*)((const bf16_t*)p + off);
    v[0] = bf2f(q.x & 0xFFFFu); v[1] = bf2f(q.x >> 16);
    v[2] = bf2f(q.y & 0xFFFFu); v[3] = bf2f(q.y >> 16);
    v[4] = bf2f(q.z & 0xFFFFu); v[5] = bf2f(q.z >> 16);
    v[6] = bf2f(q.w & 0xFFFFu); v[7] = bf2f(q.w >> 16);
  } else {
    const float4 a = *(const float4*)((const float*)p + off);
    const float4 b = *(const float4*)((const float*)p + off + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}
// load8 with streaming (non-temporal) loads, for data read exactly once
typedef unsigned int nt_u4 __attribute__((ext_vector_type(4)));
typedef float nt_f4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void load8_stream(const void* p, long long off, int bf16, float v[8]) {
  if (bf16) {
    const nt_u4 q = __builtin_nontemporal_load((const nt_u4*)((const bf16_t*)p + off));
    v[0] = bf2f(q.x & 0xFFFFu); v[1] = bf2f(q.x >> 16);
    v[2] = bf2f(q.y & 0xFFFFu); v[3] = bf2f(q.y >> 16);
    v[4] = bf2f(q.z & 0xFFFFu); v[5] = bf2f(q.z >> 16);
    v[6] = bf2f(q.w & 0xFFFFu); v[7] = bf2f(q.w >> 16);
  } else {
    const nt_f4v a = __builtin_nontemporal_load((const nt_f4v*)((const float*)p + off));
    const nt_f4v b = __builtin_nontemporal_load((const nt_f4v*)((const float*)p + off + 4));
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}
__device__ __forceinline__ void store8(void* p, long long off, int bf16, const float v[8]) {
  if (bf16) {
    uint4 q;
    q.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
    q.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
    q.z = f2bf(v[4]) | (f2bf(v[5]) << 16);
    q.w = f2bf(v[6]) | (f2bf(v[7]) << 16);
    *(uint4*)((bf16_t*)p + off) = q;
  } else {
    *(float4*)((float*)p + off) = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)((float*)p + off + 4) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// ---------------------------------------------------------------- input staging
// One thread per output pixel and 8-channel group: reads C planes (coalesced along
// w across threads), writes one 16-byte (bf16) or 32-byte (fp32) NHWC chunk.
__global__ void stage_images_kernel(const float* __restrict__ x, void* y, int N, int C, int H, int W, int Cs,
                                    int to_bf16) {
  const int groups = Cs / 8;
  const long long HW = (long long)H * W;
  const long long total = (long long)N * HW * groups;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int g = (int)(idx / (N * HW));            // group-major: neighbouring threads share g
  const long long pix = idx - (long long)g * N * HW;
  const long long n = pix / HW, hw = pix - n * HW;
  float v[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int c = g * 8 + j;
    v[j] = c < C ? x[(n * C + c) * HW + hw] : 0.f;
  }
  store8(y, pix * Cs + g * 8, to_bf16, v);
}

hipError_t launch_stage_images(const float* x, void* y, int N, int C, int H, int W, int Cs, int to_bf16,
                               hipStream_t s) {
  const long long total = (long long)N * H * W * (Cs / 8);
  launch(stage_images_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), s, x, y, N, C, H,
                     W, Cs, to_bf16);
  return hipGetLastError();
}

// ---------------------------------------------------------------- max-pool
// stream = 1 (windows do not overlap, stride >= k): every input value is read once, with
// streaming loads; overlapping windows re-read neighbours from cache and load normally.
__global__ void maxpool_kernel(GroupIO io, int N, int H, int W, int Cs, int Ho, int Wo, int k, int stride, int pad,
                               int bf16, int stream) {
  const void* __restrict__ x = io.x[blockIdx.z];
  void* y = io.y[blockIdx.z];
  const int groups = Cs / 8;
  const long long total = (long long)N * Ho * Wo * groups;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int g = (int)(idx % groups);
  const long long pix = idx / groups;
  const int wo = (int)(pix % Wo);
  const long long t = pix / Wo;
  const int ho = (int)(t % Ho);
  const long long n = t / Ho;
  float m[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m[j] = -INFINITY;
  for (int u = 0; u < k; ++u) {
    const int hi = ho * stride - pad + u;
    if (hi < 0 || hi >= H) continue;
    for (int v = 0; v < k; ++v) {
      const int wi = wo * stride - pad + v;
      if (wi < 0 || wi >= W) continue;
      float q[8];
      const long long off = ((n * H + hi) * W + wi) * Cs + g * 8;
      if (stream) load8_stream(x, off, bf16, q);
      else load8(x, off, bf16, q);
#pragma unroll
      for (int j = 0; j < 8; ++j) m[j] = fmaxf(m[j], q[j]);
    }
  }
  store8(y, pix * Cs + g * 8, bf16, m);
}

// 3x3 stride-2 windows (bf16): a thread takes one 8-channel group of two vertically
// adjacent outputs (rows 2r, 2r + 1), whose windows cover input rows 4r - pad .. 4r - pad
// + 4; all 15 loads of the 5 x 3 block are issued before any max (positions outside the
// image are clamped into it and masked out).  Max is exact, so the result is that of
// the one-output kernel above.
__global__ __launch_bounds__(256) void maxpool3s2_kernel(GroupIO io, int N, int H, int W, int G, int Ho, int Wo,
                                                         int pad) {
  const uint4* __restrict__ x = (const uint4*)io.x[blockIdx.z];
  uint4* y = (uint4*)io.y[blockIdx.z];
  const int Hr = (Ho + 1) / 2;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)N * Hr * Wo * G) return;
  const int g = (int)(idx % G);
  const long long pix = idx / G;
  const int wo = (int)(pix % Wo);
  const long long t = pix / Wo;
  const int r = (int)(t % Hr);
  const long long n = t / Hr;
  uint4 q[15];
  bool ok[15];
#pragma unroll
  for (int u = 0; u < 5; ++u)
#pragma unroll
    for (int v = 0; v < 3; ++v) {
      const int hi = 4 * r - pad + u, wi = 2 * wo - pad + v;
      ok[u * 3 + v] = hi >= 0 && hi < H && wi >= 0 && wi < W;
      const int hc = min(max(hi, 0), H - 1), wc = min(max(wi, 0), W - 1);
      q[u * 3 + v] = x[((n * H + hc) * W + wc) * G + g];
    }
  float a[8], b[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) a[j] = b[j] = -INFINITY;
#pragma unroll
  for (int u = 0; u < 5; ++u)
#pragma unroll
    for (int v = 0; v < 3; ++v) {
      if (!ok[u * 3 + v]) continue;
      const uint4 w = q[u * 3 + v];
      const float f[8] = {bf2f(w.x & 0xFFFFu), bf2f(w.x >> 16), bf2f(w.y & 0xFFFFu), bf2f(w.y >> 16),
                          bf2f(w.z & 0xFFFFu), bf2f(w.z >> 16), bf2f(w.w & 0xFFFFu), bf2f(w.w >> 16)};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (u <= 2) a[j] = fmaxf(a[j], f[j]);
        if (u >= 2) b[j] = fmaxf(b[j], f[j]);
      }
    }
  store8(y, ((n * Ho + 2 * r) * Wo + wo) * G * 8 + g * 8, 1, a);
  if (2 * r + 1 < Ho) store8(y, ((n * Ho + 2 * r + 1) * Wo + wo) * G * 8 + g * 8, 1, b);
}

hipError_t launch_maxpool(const GroupIO& io, int N, int H, int W, int Cs, int Ho, int Wo, int k, int stride, int pad,
                          int bf16, hipStream_t s) {
  if (io.n < 1 || io.n > kMaxGroup) return hipErrorInvalidValue;
  if (bf16 && k == 3 && stride == 2) {
    const long long total = (long long)N * ((Ho + 1) / 2) * Wo * (Cs / 8);
    launch(maxpool3s2_kernel, dim3((unsigned)((total + 255) / 256), 1, io.n), dim3(256), s, io, N, H, W, Cs / 8, Ho,
           Wo, pad);
    return hipGetLastError();
  }
  const long long total = (long long)N * Ho * Wo * (Cs / 8);
  launch(maxpool_kernel, dim3((unsigned)((total + 255) / 256), 1, io.n), dim3(256), s, io, N, H, W, Cs, Ho, Wo, k,
         stride, pad, bf16, stride >= k ? 1 : 0);
  return hipGetLastError();
}

// ---------------------------------------------------------------- GAP / max over time
// Block (image n, chunk of GB 8-channel groups); the 256 threads form P = 256 / GB
// position slices of GB groups.  Thread (slice s, group g) reduces positions s, s + P,
// s + 2P, ... in increasing order (four 16-byte streaming loads in flight: every input
// value is read once), then thread (0, g) folds the P partial results in slice order.
// The order is fixed, so results are deterministic; sums are fp32.
constexpr int kReduceThreads = 256;

// With branches (ReduceSegs) each of a thread's 8 channels stops at its own position
// count: positions below the smallest of the 8 counts fold unmasked, the few above it
// channel by channel; channels in no branch are not read; results go out one element
// at a time to the branch's place.  The fused branches' max runs 1024 threads per
// request (one block per request, long position ranges).
template <int THREADS>
__global__ __launch_bounds__(THREADS) void spatial_reduce_kernel(GroupIO io, int HW, int Cs, int GB, int is_max,
                                                                 int bf16, ReduceSegs sg) {
  const void* __restrict__ x = io.x[blockIdx.z];
  void* y = io.y[blockIdx.z];
  __shared__ float part[THREADS * 8];
  const int G = Cs / 8, P = THREADS / GB;
  const int t = threadIdx.x, gl = t % GB, sl = t / GB;
  const int g = blockIdx.y * GB + gl;
  const long long n = blockIdx.x;
  const float init = is_max ? -INFINITY : 0.f;
  int lim[8], dst[8];   // positions of each channel; its output channel (-1: none)
  int lo = HW, hi = HW;
  if (sg.n > 0) {
    lo = HW;
    hi = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = g * 8 + j;
      lim[j] = 0;
      dst[j] = -1;
      for (int i = 0; i < sg.n; ++i)
        if (c >= sg.src[i] && c < sg.src[i] + sg.cnt[i]) {
          lim[j] = sg.len[i];
          dst[j] = sg.dst[i] + (c - sg.src[i]);
        }
      if (dst[j] >= 0) {
        lo = min(lo, lim[j]);
        hi = max(hi, lim[j]);
      }
    }
    if (hi == 0) lo = 0;   // no channel of this group is in a branch
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (dst[j] < 0) lim[j] = lo;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      lim[j] = HW;
      dst[j] = g * 8 + j;
    }
  }
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = init;
  auto fold = [&](const float q[8]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = is_max ? fmaxf(acc[j], q[j]) : acc[j] + q[j];
  };
  if (sl < P && g < G) {
    const long long base = n * HW * Cs + g * 8;
    int p = sl;
    for (; p + 3 * P < lo; p += 4 * P) {
      float q0[8], q1[8], q2[8], q3[8];
      load8_stream(x, base + (long long)p * Cs, bf16, q0);
      load8_stream(x, base + (long long)(p + P) * Cs, bf16, q1);
      load8_stream(x, base + (long long)(p + 2 * P) * Cs, bf16, q2);
      load8_stream(x, base + (long long)(p + 3 * P) * Cs, bf16, q3);
      fold(q0); fold(q1); fold(q2); fold(q3);
    }
    for (; p < lo; p += P) {
      float q[8];
      load8_stream(x, base + (long long)p * Cs, bf16, q);
      fold(q);
    }
    for (; p < hi; p += P) {
      float q[8];
      load8_stream(x, base + (long long)p * Cs, bf16, q);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (p < lim[j]) acc[j] = is_max ? fmaxf(acc[j], q[j]) : acc[j] + q[j];
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) part[t * 8 + j] = acc[j];
  if (sg.n > 0 && blockIdx.y == 0)
    for (int c = sg.zero_from + t; c < sg.ldy; c += THREADS) {
      if (bf16) ((bf16_t*)y)[n * sg.ldy + c] = 0;
      else ((float*)y)[n * sg.ldy + c] = 0.f;
    }
  __syncthreads();
  if (sl != 0 || g >= G) return;
  for (int r = 1; r < P; ++r) {
    float q[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = part[(r * GB + gl) * 8 + j];
    fold(q);
  }
  if (!is_max) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = acc[j] * (1.0f / (float)lim[j]);
  }
  if (sg.n == 0) {
    store8(y, n * Cs + g * 8, bf16, acc);
    return;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (dst[j] < 0) continue;
    if (bf16) ((bf16_t*)y)[n * sg.ldy + dst[j]] = (bf16_t)f2bf(acc[j]);
    else ((float*)y)[n * sg.ldy + dst[j]] = acc[j];
  }
}

// Without branches and with at least 16,384 (image, 8-channel group) pairs: one thread
// per pair reduces the positions 0 .. HW - 1 in increasing order, eight 16-byte
// streaming loads in flight (fp32 sums; the order is fixed, so results are
// deterministic).  Enough pairs fill the device without splitting positions, and no
// block-level fold is needed.
template <typename T>
__global__ __launch_bounds__(256) void spatial_reduce_rows_kernel(GroupIO io, int N, int HW, int G, int is_max) {
  const T* __restrict__ x = (const T*)io.x[blockIdx.z];
  T* y = (T*)io.y[blockIdx.z];
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)N * G) return;
  const int g = (int)(idx % G);
  const long long n = idx / G;
  const bool bf = sizeof(T) == 2;
  const long long base = n * HW * (long long)G * 8 + g * 8;
  const long long step = (long long)G * 8;
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = is_max ? -INFINITY : 0.f;
  int p = 0;
  for (; p + 8 <= HW; p += 8) {
    float q[8][8];
#pragma unroll
    for (int u = 0; u < 8; ++u) load8_stream(x, base + (p + u) * step, bf, q[u]);
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = is_max ? fmaxf(acc[j], q[u][j]) : acc[j] + q[u][j];
  }
  for (; p < HW; ++p) {
    float q[8];
    load8_stream(x, base + p * step, bf, q);
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = is_max ? fmaxf(acc[j], q[j]) : acc[j] + q[j];
  }
  if (!is_max) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = acc[j] * (1.0f / (float)HW);
  }
  store8(y, n * G * 8 + g * 8, bf, acc);
}

hipError_t launch_spatial_reduce(const GroupIO& io, int N, int HW, int Cs, int is_max, int bf16, hipStream_t s,
                                 const ReduceSegs* segs) {
  if (io.n < 1 || io.n > kMaxGroup) return hipErrorInvalidValue;
  if (!segs && (long long)N * (Cs / 8) >= 16384) {
    const long long total = (long long)N * (Cs / 8);
    const dim3 grid((unsigned)((total + 255) / 256), 1, io.n);
    if (bf16) launch(spatial_reduce_rows_kernel<bf16_t>, grid, dim3(256), s, io, N, HW, Cs / 8, is_max);
    else launch(spatial_reduce_rows_kernel<float>, grid, dim3(256), s, io, N, HW, Cs / 8, is_max);
    return hipGetLastError();
  }
  ReduceSegs sg{};
  if (segs) {
    if (segs->n < 0 || segs->n > kMaxReduceSegs || segs->zero_from < 0 || segs->zero_from > segs->ldy)
      return hipErrorInvalidValue;
    for (int i = 0; i < segs->n; ++i)
      if (segs->len[i] < 1 || segs->len[i] > HW || segs->cnt[i] < 1 || segs->src[i] < 0 ||
          segs->src[i] + segs->cnt[i] > Cs || segs->dst[i] < 0 || segs->dst[i] + segs->cnt[i] > segs->zero_from)
        return hipErrorInvalidValue;
    sg = *segs;
  }
  const int G = Cs / 8;
  const int GB = G < 64 ? G : 64;
  const dim3 grid((unsigned)N, (unsigned)((G + GB - 1) / GB), io.n);
  if (sg.n > 0)
    launch(spatial_reduce_kernel<1024>, grid, dim3(1024), s, io, HW, Cs, GB, is_max, bf16, sg);
  else
    launch(spatial_reduce_kernel<kReduceThreads>, grid, dim3(kReduceThreads), s, io, HW, Cs, GB, is_max, bf16, sg);
  return hipGetLastError();
}

// ---------------------------------------------------------------- fused branches' max
__global__ void maxslot_finish_kernel(GroupIO io, int ldslot, int N, ReduceSegs sg) {
  unsigned* slot = io.slot[blockIdx.z];
  void* y = io.y[blockIdx.z];
  const int n = blockIdx.x;
  const int c = blockIdx.y * blockDim.x + threadIdx.x;
  if (n >= N || c >= sg.ldy) return;
  float v = 0.f;
  for (int i = 0; i < sg.n; ++i)
    if (c >= sg.dst[i] && c < sg.dst[i] + sg.cnt[i]) {
      unsigned* p = slot + (long long)n * ldslot + sg.src[i] + (c - sg.dst[i]);
      v = max_key_value(*p);
      *p = 0u;
    }
  ((bf16_t*)y)[(long long)n * sg.ldy + c] = (bf16_t)f2bf(v);
}

hipError_t launch_maxslot_finish(const GroupIO& io, int ldslot, int N, const ReduceSegs& sg, hipStream_t s) {
  if (sg.n < 1 || sg.n > kMaxReduceSegs || N < 1 || io.n < 1 || io.n > kMaxGroup) return hipErrorInvalidValue;
  for (int i = 0; i < sg.n; ++i)
    if (sg.cnt[i] < 1 || sg.src[i] < 0 || sg.src[i] + sg.cnt[i] > ldslot || sg.dst[i] < 0 ||
        sg.dst[i] + sg.cnt[i] > sg.zero_from || sg.zero_from > sg.ldy)
      return hipErrorInvalidValue;
  launch(maxslot_finish_kernel, dim3((unsigned)N, (unsigned)((sg.ldy + 255) / 256), io.n), dim3(256), s, io, ldslot, N,
         sg);
  return hipGetLastError();
}

// ---------------------------------------------------------------- embedding gather
__global__ void embed_gather_kernel(const int32_t* __restrict__ tok, const void* __restrict__ table, void* y,
                                    int N, int L, int Cs, int vocab, int bf16) {
  const int groups = Cs / 8;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)N * L * groups) return;
  const int g = (int)(idx % groups);
  const long long pos = idx / groups;
  const int id = tok[pos];
  const bool ok = (unsigned)id < (unsigned)vocab;
  const long long row = ok ? id : 0;
  if (bf16) {
    *((uint4*)((bf16_t*)y + pos * Cs) + g) =
        ok ? *((const uint4*)((const bf16_t*)table + row * Cs) + g) : make_uint4(0u, 0u, 0u, 0u);
  } else {
    const float4* src = (const float4*)((const float*)table + row * Cs + g * 8);
    float4* dst = (float4*)((float*)y + pos * Cs + g * 8);
    const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
    dst[0] = ok ? src[0] : z;
    dst[1] = ok ? src[1] : z;
  }
}

hipError_t launch_embed_gather(const int32_t* tok, const void* table, void* y, int N, int L, int Cs, int vocab,
                               int bf16, hipStream_t s) {
  const long long total = (long long)N * L * (Cs / 8);
  launch(embed_gather_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), s, tok, table, y, N,
                     L, Cs, vocab, bf16);
  return hipGetLastError();
}

// ---------------------------------------------------------------- concat
__global__ void concat_kernel(const void* a, int ca, int lda, const void* b, int cb, int ldb, void* y, int ldy,
                              int N, int bf16) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)N * ldy) return;
  const long long n = idx / ldy;
  const int c = (int)(idx - n * ldy);
  if (bf16) {
    bf16_t v = 0;
    if (c < ca) v = ((const bf16_t*)a)[n * lda + c];
    else if (c < ca + cb) v = ((const bf16_t*)b)[n * ldb + (c - ca)];
    ((bf16_t*)y)[idx] = v;
  } else {
    float v = 0.f;
    if (c < ca) v = ((const float*)a)[n * lda + c];
    else if (c < ca + cb) v = ((const float*)b)[n * ldb + (c - ca)];
    ((float*)y)[idx] = v;
  }
}

hipError_t launch_concat(const void* a, int ca, int lda, const void* b, int cb, int ldb, void* y, int ldy, int N,
                         int bf16, hipStream_t s) {
  const long long total = (long long)N * ldy;
  launch(concat_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), s, a, ca, lda, b, cb, ldb,
                     y, ldy, N, bf16);
  return hipGetLastError();
}

// ---------------------------------------------------------------- fp32 direct conv
// One thread per (pixel, output channel); taps outer, channels inner (fp32 FMA).
// One thread per (pixel, 4 consecutive output channels).  Weights are [Kp][Co_pad]
// (K-major), so a lane's 4 weights of one K index are one 16-byte load and the lanes
// of a wave read consecutive ones; the input chunk is shared by the lanes of a pixel.
// Each output sums its products in (u, v, ci) order with fmaf.
__global__ void conv_f32_kernel(ConvArgs a) {
  use_member(a);
  const int groups = (a.c_write + 3) / 4;
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long long)a.M * groups) return;
  const int m = (int)(idx / groups);
  const int co = 4 * (int)(idx - (long long)m * groups);
  const int HoWo = a.Ho * a.Wo;
  const int n = m / HoWo, r = m - n * HoWo;
  const int ho = r / a.Wo, wo = r - ho * a.Wo;
  const float* X = (const float*)a.x;
  const float* Wt = (const float*)a.w + co;
  float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
  for (int u = 0; u < a.kh; ++u) {
    const int hi = ho * a.stride - a.pad + u;
    if (hi < 0 || hi >= a.H) continue;
    for (int v = 0; v < a.kw; ++v) {
      const int wi = wo * a.stride - a.pad + v;
      if (wi < 0 || wi >= a.W) continue;
      const float* xp = X + (((long long)n * a.H + hi) * a.W + wi) * a.Cs;
      const float* wp = Wt + (long long)((u * a.kw + v) * a.Cs) * a.Co_pad;
      for (int ci = 0; ci < a.Cs; ci += 4) {
        const float4 x4 = *(const float4*)(xp + ci);
        const float xv[4] = {x4.x, x4.y, x4.z, x4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float4 w4 = *(const float4*)(wp + (long long)(ci + i) * a.Co_pad);
          s0 = fmaf(xv[i], w4.x, s0);
          s1 = fmaf(xv[i], w4.y, s1);
          s2 = fmaf(xv[i], w4.z, s2);
          s3 = fmaf(xv[i], w4.w, s3);
        }
      }
    }
  }
  const float sv[4] = {s0, s1, s2, s3};
  const long long o = (long long)m * a.ldy + co;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (co + j >= a.c_write) break;
    float y = sv[j] * a.scale[co + j] + a.shift[co + j];
    if (a.res) y += ((const float*)a.res)[o + j];
    if (a.relu) y = fmaxf(y, 0.f);
    ((float*)a.y)[o + j] = y;
  }
}

hipError_t launch_conv_f32(const ConvArgs& a, hipStream_t s) {
  if (a.Cs % 4 != 0 || a.Co_pad % 4 != 0 || a.c_write > a.Co_pad) return hipErrorInvalidValue;
  const long long total = (long long)a.M * ((a.c_write + 3) / 4);
  if (a.n_members > kMaxGroup) return hipErrorInvalidValue;
  launch(conv_f32_kernel, dim3((unsigned)((total + 255) / 256), 1, a.n_members > 1 ? a.n_members : 1), dim3(256), s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- ensemble combine
// One wavefront per request row.  For each selected model: row max and sum of
// exp(z - max) by butterfly reductions (fixed order, deterministic), p = e / sum
// accumulated into the lane's registers; then the mean over models and the argmax
// (largest value, lowest index on ties) by a second butterfly.
constexpr int kCombineMaxPerLane = 16;   // C <= 64 * 16 = 1024 classes

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// VEC = 4 (n_classes a multiple of 4): lane-contiguous float4 loads and stores, each
// lane holding classes 4 (i * 64 + lane) + j; VEC = 1: classes i * 64 + lane.  Either way
// the classes a lane holds increase with its register index, so keeping the first
// maximum in a lane and the lower index across lanes gives the first-index argmax.
typedef float nt_f4 __attribute__((ext_vector_type(4)));   // streaming (non-temporal) 16-byte accesses

template <int VEC>
__device__ __forceinline__ int class_of(int i, int j, int lane) {
  return VEC == 4 ? 4 * (i * 64 + lane) + j : i * 64 + lane;
}

// Loads the row's logits of one model into v (-inf past n_classes).
template <int VEC>
__device__ __forceinline__ void load_row(const float* z, int C, int lane, float v[kCombineMaxPerLane]) {
  if constexpr (VEC == 4) {
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane / 4; ++i) {
      const int c = 4 * (i * 64 + lane);
      const nt_f4 q = c < C ? __builtin_nontemporal_load((const nt_f4*)(z + c))
                            : nt_f4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      v[4 * i + 0] = q.x; v[4 * i + 1] = q.y; v[4 * i + 2] = q.z; v[4 * i + 3] = q.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane; ++i) {
      const int c = i * 64 + lane;
      v[i] = c < C ? z[c] : -INFINITY;
    }
  }
}

template <int VEC>
__global__ __launch_bounds__(256) void combine_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.n) return;
  constexpr int R = kCombineMaxPerLane / VEC;   // register groups of VEC classes
  float acc[kCombineMaxPerLane];
#pragma unroll
  for (int i = 0; i < kCombineMaxPerLane; ++i) acc[i] = 0.f;
  // the next selected model's row is loaded while this one is reduced
  float nxt[kCombineMaxPerLane];
  load_row<VEC>(a.logits + a.sel[0] * a.ld_model + (long long)row * a.C, a.C, lane, nxt);
  for (int s = 0; s < a.S; ++s) {
    float v[kCombineMaxPerLane];
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane; ++i) v[i] = nxt[i];
    if (s + 1 < a.S) load_row<VEC>(a.logits + a.sel[s + 1] * a.ld_model + (long long)row * a.C, a.C, lane, nxt);
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane; ++i) mx = fmaxf(mx, v[i]);
    mx = wave_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const int k = i * VEC + j;
        v[k] = class_of<VEC>(i, j, lane) < a.C ? expf(v[k] - mx) : 0.f;
        sum += v[k];
      }
    sum = wave_sum(sum);
    const float inv = 1.0f / sum;
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane; ++i) acc[i] += v[i] * inv;
  }
  const float invS = 1.0f / (float)a.S;
  float best = -INFINITY;
  int bidx = 0x7fffffff;
  float* prow = a.probs + (long long)row * a.C;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float p[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      p[j] = acc[i * VEC + j] * invS;
      const int c = class_of<VEC>(i, j, lane);
      if (c < a.C && p[j] > best) { best = p[j]; bidx = c; }
    }
    const int c0 = class_of<VEC>(i, 0, lane);
    if (c0 < a.C) {
      if constexpr (VEC == 4) __builtin_nontemporal_store(nt_f4{p[0], p[1], p[2], p[3]}, (nt_f4*)(prow + c0));
      else prow[c0] = p[0];
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bidx, o, 64);
    if (ob > best || (ob == best && oi < bidx)) { best = ob; bidx = oi; }
  }
  if (lane == 0) a.labels[row] = bidx;
}

// The float4 path needs every row of logits and of the output on a 16-byte boundary.
static bool vec4_ok(const CombineArgs& a) {
  return a.C % 4 == 0 && a.ld_model % 4 == 0 &&
         (((uintptr_t)a.logits | (uintptr_t)a.probs) & 15) == 0;
}

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
  if (a.C > 64 * kCombineMaxPerLane || a.S < 1) return hipErrorInvalidValue;
  if (vec4_ok(a)) launch(combine_kernel<4>, dim3((a.n + 3) / 4), dim3(256), s, a);
  else launch(combine_kernel<1>, dim3((a.n + 3) / 4), dim3(256), s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- majority vote
// One wave per request row.  Each selected model's prediction is the first index of
// the maximum of its logits; lane s keeps the prediction of selected model s (S <= 32,
// priority = selection order).  The winner is the prediction with the most votes,
// the tie going to the lowest s.  All integer work: exact and order independent.
template <int VEC>
__global__ __launch_bounds__(256) void vote_kernel(CombineArgs a) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.n) return;
  constexpr int R = kCombineMaxPerLane / VEC;
  int pred_mine = -1;
  // all of a row's loads first, then the scan; the next model's row is loaded while
  // this one is scanned
  float nxt[kCombineMaxPerLane];
  load_row<VEC>(a.logits + a.sel[0] * a.ld_model + (long long)row * a.C, a.C, lane, nxt);
  for (int s = 0; s < a.S; ++s) {
    float v[kCombineMaxPerLane];
#pragma unroll
    for (int i = 0; i < kCombineMaxPerLane; ++i) v[i] = nxt[i];
    if (s + 1 < a.S) load_row<VEC>(a.logits + a.sel[s + 1] * a.ld_model + (long long)row * a.C, a.C, lane, nxt);
    float best = -INFINITY;
    int bidx = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int j = 0; j < VEC; ++j)
        if (v[i * VEC + j] > best) { best = v[i * VEC + j]; bidx = class_of<VEC>(i, j, lane); }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ob = __shfl_xor(best, o, 64);
      const int oi = __shfl_xor(bidx, o, 64);
      if (ob > best || (ob == best && oi < bidx)) { best = ob; bidx = oi; }
    }
    if (bidx == 0x7fffffff) bidx = 0;        // a row with no value above -inf
    if (lane == s) pred_mine = bidx;
  }
  // one broadcast per model's prediction: the votes for this lane's prediction, and
  // for each class this lane writes
  int count = 0;
  int votes[kCombineMaxPerLane];
#pragma unroll
  for (int e = 0; e < kCombineMaxPerLane; ++e) votes[e] = 0;
  for (int t = 0; t < a.S; ++t) {
    const int p = __shfl(pred_mine, t, 64);
    count += p == pred_mine ? 1 : 0;
#pragma unroll
    for (int i = 0; i < R; ++i)
#pragma unroll
      for (int j = 0; j < VEC; ++j) votes[i * VEC + j] += class_of<VEC>(i, j, lane) == p ? 1 : 0;
  }
  int key = lane < a.S ? count * 64 + (63 - lane) : -1;   // most votes, then lowest s
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) key = max(key, __shfl_xor(key, o, 64));
  const int winner = 63 - (key & 63);
  const int label = __shfl(pred_mine, winner, 64);
  const float invS = 1.0f / (float)a.S;
  float* prow = a.probs + (long long)row * a.C;
#pragma unroll
  for (int i = 0; i < R; ++i) {
    float f[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) f[j] = (float)votes[i * VEC + j] * invS;
    const int c0 = class_of<VEC>(i, 0, lane);
    if (c0 < a.C) {
      if constexpr (VEC == 4) __builtin_nontemporal_store(nt_f4{f[0], f[1], f[2], f[3]}, (nt_f4*)(prow + c0));
      else prow[c0] = f[0];
    }
  }
  if (lane == 0) a.labels[row] = label;
}

hipError_t launch_vote(const CombineArgs& a, hipStream_t s) {
  if (a.S < 1 || a.S > 32 || a.C < 1 || a.C > 64 * kCombineMaxPerLane) return hipErrorInvalidValue;
  if (vec4_ok(a)) launch(vote_kernel<4>, dim3((a.n + 3) / 4), dim3(256), s, a);
  else launch(vote_kernel<1>, dim3((a.n + 3) / 4), dim3(256), s, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------- peak probes
// Matrix-core ceiling: each wave keeps 8 independent 32x32 fp32 accumulators and
// issues `iters` rounds of 8 v_mfma_f32_32x32x16_bf16 on register-resident operands
// (nothing is loaded inside the loop); one checksum per wave keeps the work alive.
typedef __bf16 probe_bf16x8 __attribute__((ext_vector_type(8)));
typedef float probe_f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void probe_mfma_kernel(int iters, float* out) {
  probe_bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((threadIdx.x + i) & 7));
    b[i] = (__bf16)(0.002f * (float)((threadIdx.x * 3 + i) & 7));
  }
  probe_f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float t = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) t += acc[j][e];
  if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = t;
}

hipError_t launch_probe_mfma(int blocks, int iters, float* out, hipStream_t s) {
  launch(probe_mfma_kernel, dim3(blocks), dim3(256), s, iters, out);
  return hipGetLastError();
}

// HBM read ceiling: a grid-stride pass of 16-byte streaming loads over `words16`
// 16-byte words, folded into one value per block.
typedef unsigned probe_u4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void probe_read_kernel(const probe_u4* __restrict__ x, long long words16,
                                                         unsigned* out) {
  unsigned acc = 0;
  const long long stride = (long long)gridDim.x * blockDim.x;
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < words16; i += 4 * stride) {
    const probe_u4 v0 = __builtin_nontemporal_load(x + i), v1 = __builtin_nontemporal_load(x + i + stride);
    const probe_u4 v2 = __builtin_nontemporal_load(x + i + 2 * stride);
    const probe_u4 v3 = __builtin_nontemporal_load(x + i + 3 * stride);
    const probe_u4 v = v0 ^ v1 ^ v2 ^ v3;
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  for (; i < words16; i += stride) {
    const probe_u4 v = __builtin_nontemporal_load(x + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = acc;
}

hipError_t launch_probe_read(const void* x, long long words16, int blocks, unsigned* out, hipStream_t s) {
  launch(probe_read_kernel, dim3(blocks), dim3(256), s, (const probe_u4*)x, words16, out);
  return hipGetLastError();
}

// Main-loop skeleton of the GEMM kernel, nothing loaded from memory: per K tile of 64,
// four k-steps in which each wave reads its TM + TN fragments from LDS (the conv
// kernel's conflict-free swizzle; the next step's reads issued ahead of this step's
// MFMAs) and runs its TM x TN v_mfma_f32_32x32x16_bf16.  With SYNC each K tile also
// writes the tile's volume, (BM + BN) rows x 64 bf16, into LDS from registers and passes
// a workgroup barrier, as the refill of a stage does.  Every LDS index stays inside the
// 80 KB array: fragment rows r < 256 of 8 chunks for each operand, writes to the last
// 1024 chunks.  The addresses alternate with the tile so that no read is loop-invariant.
template <int NW, int WM, int TM, int TN, bool SYNC>
__global__ __launch_bounds__(NW * 64, 1) void probe_mainloop_kernel(int ktiles, float* out) {
  __shared__ probe_u4 lds[5120];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // bf16 values in [2^-7, 2^-6): sums over any number of tiles here stay finite
  for (int i = tid; i < 5120; i += NW * 64) {
    const unsigned u = (unsigned)i;
    lds[i] = probe_u4{0x3C003C00u | (u & 0x7F) | ((3 * u & 0x7F) << 16), 0x3C003C00u | (5 * u & 0x7F),
                      0x3C003C00u | ((7 * u & 0x7F) << 16), 0x3C003C00u | (11 * u & 0x7F)};
  }
  __syncthreads();
  probe_f32x16 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  const int frow = lane & 31, fk = lane >> 5;
  const int wm = wave % WM, wn = wave / WM;
  auto frag = [&](int base, int r, int kc) {
    r &= 255;
    return __builtin_bit_cast(probe_bf16x8, lds[base + r * 8 + (kc ^ (r & 7) ^ ((r >> 3) & 1))]);
  };
  probe_bf16x8 xf[2][TM], wf[2][TN];
#pragma unroll
  for (int tm = 0; tm < TM; ++tm) xf[0][tm] = frag(0, wm * 32 * TM + tm * 32 + frow, fk);
#pragma unroll
  for (int tn = 0; tn < TN; ++tn) wf[0][tn] = frag(2048, wn * 32 * TN + tn * 32 + frow, fk);
  for (int kt = 0; kt < ktiles; ++kt) {
    const int ro = (kt & 1) * 32;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const int b = st & 1, nx = 2 * ((st + 1) & 3) + fk;
#pragma unroll
      for (int tm = 0; tm < TM; ++tm) xf[b ^ 1][tm] = frag(0, ro + wm * 32 * TM + tm * 32 + frow, nx);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn) wf[b ^ 1][tn] = frag(2048, ro + wn * 32 * TN + tn * 32 + frow, nx);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tn = 0; tn < TN; ++tn)
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[b][tn], xf[b][tm], acc[tn][tm], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (SYNC) {
      constexpr int BM = 32 * TM * WM, BN = 32 * TN * (NW / WM);
      constexpr int PT = (BM + BN) * 8 / (NW * 64);   // 16-byte chunks per thread
#pragma unroll
      for (int i = 0; i < PT; ++i)
        lds[4096 + ((i * NW * 64 + tid) & 1023)] = probe_u4{(unsigned)kt, (unsigned)i, (unsigned)tid, 1u};
      __syncthreads();
    }
  }
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) t += acc[i][j][e];
  if (lane == 0) out[blockIdx.x * 8 + wave] = t;
}

// Variants: 0 = 8 waves of 64x128 (the 256x256 tile's layout), 1 = 4 waves of 128x128,
// 2 = 4 waves of 64x64 (128x128 tile), 3 = 8 waves of 64x32 (128x128 tile).
hipError_t launch_probe_mainloop(int variant, bool sync, int blocks, int ktiles, float* out, hipStream_t s) {
#define RAFIKI_PROBE_ML(NW, WM, TM, TN)                                                              \
  if (sync) launch(probe_mainloop_kernel<NW, WM, TM, TN, true>, dim3(blocks), dim3(NW * 64), s, ktiles, out); \
  else launch(probe_mainloop_kernel<NW, WM, TM, TN, false>, dim3(blocks), dim3(NW * 64), s, ktiles, out);
  switch (variant) {
    case 0: RAFIKI_PROBE_ML(8, 4, 2, 4) break;
    case 1: RAFIKI_PROBE_ML(4, 2, 4, 4) break;
    case 2: RAFIKI_PROBE_ML(4, 2, 2, 2) break;
    case 3: RAFIKI_PROBE_ML(8, 2, 2, 1) break;
    default: return hipErrorInvalidValue;
  }
#undef RAFIKI_PROBE_ML
  return hipGetLastError();
}

}  // namespace rafiki
