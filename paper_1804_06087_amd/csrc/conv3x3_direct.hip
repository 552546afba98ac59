// Direct 3x3 convolution (stride 1, zero padding 1) of bf16 NHWC layers with 64 input
// and 64 output channels on gfx950 matrix cores, optionally with the 2x2 stride-2
// max-pool fused (the conv layers of a network's full-resolution stage: VGG-16's
// conv1_2, the 56x56 3x3 layers of ResNet-50/101; Section 5.1, each model's forward
// pass over the batch).
//
// Why a kernel of its own: the implicit GEMM brings every input pixel into LDS nine
// times, once per tap, and with only 64 output channels each 16-byte chunk it loads
// feeds just two MFMAs, so these layers are bound by the L2 -> LDS load path.  Here a
// persistent workgroup (one per compute unit) keeps the layer's weights (64 x 576 bf16,
// 72 KB) in LDS for its whole life, and two input patches of 18 x 18 pixels (a 16 x 16
// output tile plus the halo): the nine taps read the patch in place, and the next
// patch loads while the current one is computed.
//
// The sums are formed exactly as conv_mfma_kernel forms them for this layer: K in the
// packed order (tap u * 3 + v, then channel), 36 k-steps of v_mfma_f32_32x32x16_bf16
// in increasing K with the weights as A operand and the pixels as B operand, lane l
// holding k-range 8 * (l / 32) .. +8 of row l % 32; then fma(acc, scale, shift), the
// fp32 max over each 2x2 window when pooling, integer-max ReLU and one rounding to
// bf16.  The outputs are therefore bitwise those of the GEMM kernel, whatever its tile.
#include <algorithm>
#include <atomic>

#include "kernels.h"

namespace rafiki {
namespace {

typedef __bf16 d3_bf16x8 __attribute__((ext_vector_type(8)));
typedef float d3_f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void d3_lds_void;
typedef __bf16 d3_bf16x2 __attribute__((ext_vector_type(2)));
typedef float d3_f32x2 __attribute__((ext_vector_type(2)));

constexpr int kTile = 16;                     // output tile: 16 x 16 pixels
constexpr int kPatch = kTile + 2;             // input patch side with the halo
constexpr int kPatchPix = kPatch * kPatch;    // 324
constexpr int kPatchLoads = (kPatchPix + 7) / 8;   // one load instruction moves 8 pixels
constexpr int kPatchChunks = kPatchLoads * 64;     // 16-byte chunks per patch buffer (328 pixels)
constexpr int kWChunks = 9 * 64 * 8;               // weights: [tap][channel][8 chunks]
constexpr int kLdsChunks = kWChunks + 2 * kPatchChunks;
constexpr int kDepth = 3;   // k-steps of fragment reads in flight ahead of the MFMAs
static_assert(kLdsChunks * 16 <= 160 * 1024, "LDS budget");

// Row r keeps logical 16-byte chunk q in slot q ^ swz(r): over any 16 consecutive rows
// (r % 2, slot) is distinct, so a ds_read_b128 of one chunk from 16 consecutive rows is
// bank-conflict free.  Patch pixels are rows here, as are weight rows (channels).
__device__ __forceinline__ int d3_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

__device__ __forceinline__ uint32_t d3_pack2(float a, float b) {   // nearest even, a low
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(d3_f32x2{a, b}, d3_bf16x2));
}
__device__ __forceinline__ float d3_relu(float v) { return __int_as_float(max(__float_as_int(v), 0)); }

template <int N>
__device__ __forceinline__ void d3_wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Tile t: image t / per_img, tile row (t % per_img) / tw, tile column (t % per_img) % tw.
struct TileGeo {
  int n, oh0, ow0;
};
__device__ __forceinline__ TileGeo tile_geo(int t, int per_img, int tw) {
  const int n = t / per_img, r = t - n * per_img, th = r / tw;
  return {n, th * kTile, (r - th * tw) * kTile};
}

}  // namespace

__global__ __launch_bounds__(256, 1) void conv3x3_direct_kernel(ConvArgs a) {
  __shared__ uint4 lds[kLdsChunks];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, (short)0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, a.w_bytes, 0x00020000);
  const unsigned oob = (unsigned)a.x_bytes;   // offset at num_records: the hardware returns zeros
  const int tw = (a.W + kTile - 1) / kTile, per_img = ((a.H + kTile - 1) / kTile) * tw;
  const int ntiles = a.N * per_img;
  const int G = gridDim.x;

  // Weights, once: load i moves tap i / 8, channels 8 * (i % 8) .. +8 (all 8 chunks);
  // lane l carries chunk (l % 8) ^ swz(channel) into slot l % 8 of row (tap, channel).
  for (int i = wave; i < 72; i += 4) {
    const int t = i >> 3, co = (i & 7) * 8 + (lane >> 3);
    const int q = (lane & 7) ^ d3_swz(co);
    const unsigned off = (unsigned)((co * a.Kp + t * 64 + q * 8) * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (d3_lds_void*)(lds + i * 64), 16, off, 0, 0, 0);
  }
  // Patch of tile t into buffer b: load i moves patch pixels 8i .. 8i + 7 (pixel p is
  // input row oh0 - 1 + p / 18, column ow0 - 1 + p % 18); pixels outside the image, and
  // the 4 past the patch, read zeros.
  auto load_patch = [&](int t, int b) {
    const TileGeo g = tile_geo(t, per_img, tw);
    uint4* base = lds + kWChunks + b * kPatchChunks;
    for (int i = wave; i < kPatchLoads; i += 4) {
      const int p = i * 8 + (lane >> 3);
      const int ph = p / kPatch, pw = p - ph * kPatch;
      const int hi = g.oh0 - 1 + ph, wi = g.ow0 - 1 + pw;
      const int q = (lane & 7) ^ d3_swz(p);
      const bool ok = p < kPatchPix && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
      const unsigned off = ok ? (unsigned)((((g.n * a.H + hi) * a.W + wi) * 64 + q * 8) * 2) : oob;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (d3_lds_void*)(base + i * 64), 16, off, 0, 0, 0);
    }
  };

  const int frow = lane & 31, fk = lane >> 5;
  // Wave w computes tile rows 4w .. 4w + 3, all 64 channels; pixel block tm covers rows
  // 4w + 2tm and 4w + 2tm + 1.  Column frow of a block is the pixel at row offset
  // (frow >> 1) & 1, column 2 (frow >> 2) + (frow & 1): the four pixels of each 2x2
  // window sit in four adjacent lanes (a DPP quad).  Which pixel a column holds does
  // not change its sum.
  const int prow = (frow >> 1) & 1, pcol = 2 * (frow >> 2) + (frow & 1);
  int pix0[2];   // patch pixel of this lane's output in block tm under tap (0, 0)
#pragma unroll
  for (int tm = 0; tm < 2; ++tm) pix0[tm] = (4 * wave + 2 * tm + prow) * kPatch + pcol;
  // scale and shift of this lane's output channels tn * 32 + 8q + 4fk + j, kept in
  // registers for the workgroup's life
  float4 sc[2][4], sh[2][4];
#pragma unroll
  for (int tn = 0; tn < 2; ++tn)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sc[tn][q] = *(const float4*)(a.scale + tn * 32 + 8 * q + 4 * fk);
      sh[tn][q] = *(const float4*)(a.shift + tn * 32 + 8 * q + 4 * fk);
    }

  int t = blockIdx.x;
  if (t < ntiles) load_patch(t, 0);
  d3_wait_vmcnt<0>();
  __syncthreads();
  for (int it = 0; t < ntiles; ++it, t += G) {
    const int b = it & 1;
    if (t + G < ntiles) load_patch(t + G, b ^ 1);
    const uint4* P = lds + kWChunks + b * kPatchChunks;

    d3_f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // Fragments run kDepth k-steps ahead of the MFMAs (ring of kDepth + 1 register
    // sets): with one wave per SIMD nothing else hides the LDS latency, which under the
    // four waves' reads is about three k-steps of MFMAs.
    d3_bf16x8 xf[kDepth + 1][2], wf[kDepth + 1][2];
    // fragments of k-step ks (tap ks / 4, channels 16 * (ks % 4) .. +16) into set s
    auto rd = [&](int ks, int s) {
      const int tap = ks >> 2, u = tap / 3, v = tap - 3 * u;
      const int q = 2 * (ks & 3) + fk;
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        const int p = pix0[tm] + u * kPatch + v;
        xf[s][tm] = __builtin_bit_cast(d3_bf16x8, P[p * 8 + (q ^ d3_swz(p))]);
      }
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        const int co = tn * 32 + frow;
        wf[s][tn] = __builtin_bit_cast(d3_bf16x8, lds[(tap * 64 + co) * 8 + (q ^ d3_swz(co))]);
      }
    };
#pragma unroll
    for (int ks = 0; ks < kDepth; ++ks) rd(ks, ks);
#pragma unroll
    for (int ks = 0; ks < 36; ++ks) {
      const int s = ks % (kDepth + 1);
      if (ks + kDepth < 36) rd(ks + kDepth, (ks + kDepth) % (kDepth + 1));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tn = 0; tn < 2; ++tn)
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[s][tn], xf[s][tm], acc[tn][tm], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // This wave's loads of the next patch have landed, and every wave is done with P:
    // the next iteration may compute from the other buffer and refill this one.
    d3_wait_vmcnt<0>();
    __syncthreads();

    // Epilogue from the accumulators: lane (frow, fk) holds, for block (tn, tm),
    // channels tn * 32 + 8g + 4fk + j (g, j in 0..3) of its pixel.
    const TileGeo g = tile_geo(t, per_img, tw);
#pragma unroll
    for (int tn = 0; tn < 2; ++tn) {
#pragma unroll
      for (int tm = 0; tm < 2; ++tm) {
        const int oh = g.oh0 + 4 * wave + 2 * tm + prow, ow = g.ow0 + pcol;
        float v[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[4 * q + 0] = __builtin_fmaf(acc[tn][tm][4 * q + 0], sc[tn][q].x, sh[tn][q].x);
          v[4 * q + 1] = __builtin_fmaf(acc[tn][tm][4 * q + 1], sc[tn][q].y, sh[tn][q].y);
          v[4 * q + 2] = __builtin_fmaf(acc[tn][tm][4 * q + 2], sc[tn][q].z, sh[tn][q].z);
          v[4 * q + 3] = __builtin_fmaf(acc[tn][tm][4 * q + 3], sc[tn][q].w, sh[tn][q].w);
        }
        if (a.pool2) {
          // max over the window's quad of lanes (DPP quad_perm [1,0,3,2], then [2,3,0,1])
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            v[e] = fmaxf(v[e], __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[e]), 0xB1, 0xF, 0xF, false)));
            v[e] = fmaxf(v[e], __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[e]), 0x4E, 0xF, 0xF, false)));
          }
          if ((frow & 3) != 0 || oh >= a.H || ow >= a.W) continue;
          if (a.relu) {
#pragma unroll
            for (int e = 0; e < 16; ++e) v[e] = d3_relu(v[e]);
          }
          bf16_t* y = (bf16_t*)a.y + ((long long)(g.n * (a.H >> 1) + (oh >> 1)) * (a.W >> 1) + (ow >> 1)) * a.ldy;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *(uint2*)(y + tn * 32 + 8 * q + 4 * fk) =
                make_uint2(d3_pack2(v[4 * q], v[4 * q + 1]), d3_pack2(v[4 * q + 2], v[4 * q + 3]));
        } else {
          if (oh >= a.H || ow >= a.W) continue;
          if (a.relu) {
#pragma unroll
            for (int e = 0; e < 16; ++e) v[e] = d3_relu(v[e]);
          }
          bf16_t* y = (bf16_t*)a.y + ((long long)(g.n * a.H + oh) * a.W + ow) * a.ldy;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            *(uint2*)(y + tn * 32 + 8 * q + 4 * fk) =
                make_uint2(d3_pack2(v[4 * q], v[4 * q + 1]), d3_pack2(v[4 * q + 2], v[4 * q + 3]));
        }
      }
    }
  }
}

bool conv3x3_direct_fits(const ConvArgs& a) {
  return a.kh == 3 && a.kw == 3 && a.stride == 1 && a.pad == 1 && a.Cs == 64 && a.K == 576 && a.Kp == 576 &&
         a.Nc == 64 && a.Co_pad >= 64 && a.c_write == 64 && a.ldy >= 64 && a.ldy % 4 == 0 && a.Ho == a.H &&
         a.Wo == a.W && a.res == nullptr && !a.out_f32 && a.tap_stride == 0 && a.maxslot == nullptr &&
         a.n_members <= 1 && (!a.pool2 || (a.H % 2 == 0 && a.W % 2 == 0)) && a.N >= 1;
}

hipError_t launch_conv3x3_direct(const ConvArgs& a, hipStream_t s) {
  if (!conv3x3_direct_fits(a)) return hipErrorInvalidValue;
  // compute units per device, queried once (concurrent first calls store the same value)
  static std::atomic<int> cus[64];
  int dev = 0;
  hipError_t st = hipGetDevice(&dev);
  if (st != hipSuccess) return st;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  int n_cu = cus[dev].load(std::memory_order_relaxed);
  if (n_cu <= 0) {
    st = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (st != hipSuccess) return st;
    n_cu = n_cu > 0 ? n_cu : 1;
    cus[dev].store(n_cu, std::memory_order_relaxed);
  }
  const long long tiles = (long long)a.N * ((a.H + kTile - 1) / kTile) * ((a.W + kTile - 1) / kTile);
  const int grid = (int)std::min<long long>(tiles, n_cu);
  launch(conv3x3_direct_kernel, dim3(grid), dim3(256), s, a);
  return hipGetLastError();
}

}  // namespace rafiki
