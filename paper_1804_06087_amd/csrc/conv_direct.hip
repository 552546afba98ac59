// Direct convolution of bf16 NHWC layers with 64 output channels (or 128, as two halves)
// on gfx950 matrix cores, for the layers where the implicit GEMM is bound by its loads
// (Section 5.1, each model's forward pass over the batch):
//   - 3x3, stride 1, 64 input channels (VGG-16's conv1_2 with its fused 2x2 max-pool and
//     conv2_1, the 56x56 3x3 layers of ResNet-50/101): the GEMM brings every input pixel
//     into LDS nine times, once per tap, and with 64 output channels each 16-byte chunk
//     it loads feeds just two MFMAs;
//   - 3x3, stride 1, and 7x7, stride 2, on the 8 storage channels of an RGB image (VGG-16's
//     conv1_1, the ResNet stems): 9 or 49 taps re-read each pixel as often.
// A persistent workgroup (one or two per compute unit) keeps the layer's weights in LDS
// for its whole life, and two input patches (a 16 x 16 output tile plus its halo): the
// taps read the patch in place, and the next tile's patch loads while the current one is
// computed.
//
// The sums are formed exactly as conv_mfma_kernel forms them for these layers: K in the
// packed order (tap u * kw + v, then channel), k-steps of v_mfma_f32_32x32x16_bf16 in
// increasing K with the weights as A operand and the pixels as B operand, lane l holding
// k-range 8 * (l / 32) .. +8 of row l % 32 (with 8 channels, k-step s covers taps 2s and
// 2s + 1; a tap past the last is zero on both sides); then fma(acc, scale, shift), the
// max over each 2x2 window when pooling, integer-max ReLU and one rounding to bf16 (with
// ReLU and pool, ReLU on each value and then the integer max, which equals ReLU of the
// fp32 max for every non-NaN sum).  The outputs are therefore bitwise those of the GEMM
// kernel, whatever its tile.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "kernels.h"

namespace rafiki {
namespace {

typedef __bf16 d3_bf16x8 __attribute__((ext_vector_type(8)));
typedef float d3_f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void d3_lds_void;
typedef __bf16 d3_bf16x2 __attribute__((ext_vector_type(2)));
typedef float d3_f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned d3_u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned d3_u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = 16;    // output tile: 16 x 16 pixels
constexpr int kDepth = 3;    // k-steps of fragment reads in flight ahead of the MFMAs

// Geometry of one instance: CS storage input channels (64 or 8), KS x KS taps, stride ST.
template <int CS, int KS, int ST>
struct DGeo {
  static constexpr int CC = CS / 8;                         // 16-byte chunks per pixel
  static constexpr int PAD = KS / 2;
  static constexpr int PS = (kTile - 1) * ST + KS;          // patch side
  static constexpr int PPIX = PS * PS;
  static constexpr int PIX_PER_LOAD = 64 / CC;              // one load instruction: 64 chunks
  static constexpr int PLOADS = (PPIX + PIX_PER_LOAD - 1) / PIX_PER_LOAD;
  static constexpr int PCHUNKS = PLOADS * 64;               // per patch buffer
  static constexpr int TAPS = KS * KS;
  static constexpr int NK = (TAPS * CS + 15) / 16;          // k-steps of 16
  static constexpr int WTAPS = CS == 64 ? TAPS : 2 * NK;    // weight rows per channel (8 channels: even)
  static constexpr int WCHUNKS = WTAPS * 64 * CC;           // weights: [tap][channel][CC chunks]
  static constexpr int ZERO = WCHUNKS + 2 * PCHUNKS;        // one zero chunk (taps past the last)
  // 8 channels: each wave's 64 output pixels x 8 chunks, staged for whole-pixel stores
  static constexpr int STG = ZERO + 1;
  static constexpr int LDS_CHUNKS = STG + (CS == 8 ? 4 * 64 * 8 : 0);
  static_assert(CS == 64 || CS == 8, "64 or 8 input channels");
  static_assert(LDS_CHUNKS * 16 <= 160 * 1024, "LDS budget");
};

// Row r keeps logical 16-byte chunk q in slot q ^ swz(r): over any 16 consecutive rows
// (r % 2, slot) is distinct, so a ds_read_b128 of one chunk from 16 consecutive rows is
// bank-conflict free.  Patch pixels are rows here, as are weight rows (channels).  With
// one chunk per row (8 channels) rows are 16 bytes apart and need no swizzle.
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

template <int CS, int KS, int ST, int OCC>
__global__ __launch_bounds__(256, OCC) void conv_direct_kernel(ConvArgs a) {
  using D = DGeo<CS, KS, ST>;
  __shared__ uint4 lds[D::LDS_CHUNKS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, (short)0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.w, (short)0, a.w_bytes, 0x00020000);
  const unsigned oob = (unsigned)a.x_bytes;   // offset at num_records: the hardware returns zeros
  // Output through a buffer resource as well: the launcher takes only outputs below
  // 4 GiB, so byte offsets fit 32 bits, and an offset at num_records (yoob) is dropped.
  const int Hy = a.pool2 ? a.Ho >> 1 : a.Ho, Wy = a.pool2 ? a.Wo >> 1 : a.Wo;
  const unsigned yoob = (unsigned)((unsigned long long)a.N * Hy * Wy * a.ldy * 2);
  const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(a.y, (short)0, (int)yoob, 0x00020000);
  const int tw = (a.Wo + kTile - 1) / kTile, per_img = ((a.Ho + kTile - 1) / kTile) * tw;
  const int ntiles = a.N * per_img;
  // 64-channel input with 128 output channels: workgroup b computes the 64-channel half
  // h = b % 2 of its tiles (weights, scale, shift and outputs offset by 64 h)
  const int NH = CS == 64 ? a.Nc / 64 : 1;
  const int h = (int)blockIdx.x % NH, c0 = 64 * h;
  const int G = gridDim.x / NH;

  // Weights, once.  64 channels: load i moves tap i / 8, channels 8 * (i % 8) .. +8 (all
  // 8 chunks), lane l carrying chunk (l % 8) ^ swz(channel) into slot l % 8 of row (tap,
  // channel).  8 channels: load i moves tap i of the 64 channels, one chunk each (the
  // padded taps read the packed array's zeros).
  if constexpr (CS == 64) {
    for (int i = wave; i < D::TAPS * 8; i += 4) {
      const int t = i >> 3, co = (i & 7) * 8 + (lane >> 3);
      const int q = (lane & 7) ^ d3_swz(co);
      const unsigned off = (unsigned)(((c0 + co) * a.Kp + t * 64 + q * 8) * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (d3_lds_void*)(lds + i * 64), 16, off, 0, 0, 0);
    }
  } else {
    for (int i = wave; i < D::WTAPS; i += 4) {
      const unsigned off = (unsigned)((lane * a.Kp + i * 8) * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (d3_lds_void*)(lds + i * 64), 16, off, 0, 0, 0);
    }
  }
  if (tid == 0) lds[D::ZERO] = make_uint4(0u, 0u, 0u, 0u);

  // Patch of a tile: patch pixel p is input row oh0 * ST - PAD + p / PS, column
  // ow0 * ST - PAD + p % PS; pixels outside the image, and those past the patch, read
  // zeros.  Wave w issues loads i = w + 4j; a lane's patch row, column and offset within
  // the image are the same for every tile (a pixel past the patch gets a row that fails
  // the bounds check), so a load costs a few adds and compares.
  constexpr int kLoads = (D::PLOADS + 3) / 4;   // loads per wave and patch
  int lph[kLoads], lpw[kLoads], loff[kLoads];
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int i = wave + 4 * j;
    const int p = i * D::PIX_PER_LOAD + lane / D::CC;
    const int ph = p / D::PS, pw = p - ph * D::PS;
    lph[j] = i < D::PLOADS && p < D::PPIX ? ph : 0x40000000;
    lpw[j] = pw;
    if constexpr (CS == 64) loff[j] = (ph * a.W + pw) * 128 + ((lane & 7) ^ d3_swz(p)) * 16;
    else loff[j] = (ph * a.W + pw) * 16;
  }
  auto load_one = [&](const TileGeo& g, int b, int j) {
    const int i = wave + 4 * j;
    if (i >= D::PLOADS) return;
    const int h0 = g.oh0 * ST - D::PAD, w0 = g.ow0 * ST - D::PAD;
    const int base = ((g.n * a.H + h0) * a.W + w0) * (CS * 2);
    const bool ok = (unsigned)(h0 + lph[j]) < (unsigned)a.H && (unsigned)(w0 + lpw[j]) < (unsigned)a.W;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (d3_lds_void*)(lds + D::WCHUNKS + b * D::PCHUNKS + i * 64), 16,
                                             ok ? (unsigned)(base + loff[j]) : oob, 0, 0, 0);
  };

  const int frow = lane & 31, fk = lane >> 5;
  // Wave w computes tile rows 4w .. 4w + 3, all 64 channels (of its half).  Column frow
  // of pixel block tm is the pixel at tile row 4w + 2 (frow / 16) + tm, column frow % 16:
  // the two rows of each 2x2 window sit in one lane (blocks 0 and 1), its two columns in
  // adjacent lanes.  Which pixel a column holds does not change its sum.
  const int prow = 4 * wave + 2 * (frow >> 4), pcol = frow & 15;
  int pix0[2];   // patch pixel under tap (0, 0) of this lane's output in block tm
#pragma unroll
  for (int tm = 0; tm < 2; ++tm) pix0[tm] = (prow + tm) * ST * D::PS + pcol * ST;
  // scale and shift of this lane's output channels tn * 32 + 8q + 4fk + j, kept in
  // registers for the workgroup's life
  float4 sc[2][4], sh[2][4];
#pragma unroll
  for (int tn = 0; tn < 2; ++tn)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      sc[tn][q] = *(const float4*)(a.scale + c0 + tn * 32 + 8 * q + 4 * fk);
      sh[tn][q] = *(const float4*)(a.shift + c0 + tn * 32 + 8 * q + 4 * fk);
    }
  // Byte offsets within a tile's output, per lane: the pooled pixel of a window's
  // leading lane, or the pixel and 8-channel chunk of a whole-pixel store (8 lanes per
  // pixel, the store of step r covering tile row 4w + 2 ((r % 4) / 2) + r / 4 and columns
  // 8 (r % 2) .. + 8).
  const int ylane = a.pool2 ? ((frow >> 4) * Wy + (pcol >> 1)) * a.ldy * 2 + (c0 + 4 * fk) * 2
                            : ((lane >> 3) * a.ldy + c0 + (lane & 7) * 8) * 2;

  int t = blockIdx.x / NH;
  if (t < ntiles) {
    const TileGeo g = tile_geo(t, per_img, tw);
#pragma unroll
    for (int j = 0; j < kLoads; ++j) load_one(g, 0, j);
  }
  d3_wait_vmcnt<0>();
  __syncthreads();
  for (int it = 0; t < ntiles; ++it, t += G) {
    const int b = it & 1;
    const int pbase = D::WCHUNKS + b * D::PCHUNKS;   // the patch being computed
    // the next tile's patch goes into the other buffer, its loads spread over the k-steps
    const bool more = t + G < ntiles;
    const TileGeo gn = tile_geo(more ? t + G : t, per_img, tw);

    d3_f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // Fragments run kDepth k-steps ahead of the MFMAs (ring of kDepth + 1 register
    // sets): with one wave per SIMD nothing else hides the LDS latency.
    d3_bf16x8 xf[kDepth + 1][2], wf[kDepth + 1][2];
    // fragments of k-step ks into set s
    auto rd = [&](int ks, int s) {
      if constexpr (CS == 64) {   // tap ks / 4, channels 16 * (ks % 4) .. +16
        const int tap = ks >> 2, u = tap / KS, v = tap - KS * u;
        const int q = 2 * (ks & 3) + fk;
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
          const int p = pix0[tm] + u * D::PS + v;
          xf[s][tm] = __builtin_bit_cast(d3_bf16x8, lds[pbase + p * 8 + (q ^ d3_swz(p))]);
        }
#pragma unroll
        for (int tn = 0; tn < 2; ++tn) {
          const int co = tn * 32 + frow;
          wf[s][tn] = __builtin_bit_cast(d3_bf16x8, lds[(tap * 64 + co) * 8 + (q ^ d3_swz(co))]);
        }
      } else {   // taps 2 ks (lanes fk = 0) and 2 ks + 1 (fk = 1), 8 channels each
        const int t0 = 2 * ks, t1 = 2 * ks + 1;
        const int o0 = (t0 / KS) * D::PS + t0 % KS, o1 = (t1 / KS) * D::PS + t1 % KS;
        const bool real = fk ? t1 < D::TAPS : t0 < D::TAPS;
        const int off = fk ? o1 : o0;
#pragma unroll
        for (int tm = 0; tm < 2; ++tm) {
          const int idx = real ? pbase + pix0[tm] + off : D::ZERO;
          xf[s][tm] = __builtin_bit_cast(d3_bf16x8, lds[idx]);
        }
#pragma unroll
        for (int tn = 0; tn < 2; ++tn)
          wf[s][tn] = __builtin_bit_cast(d3_bf16x8, lds[(2 * ks + fk) * 64 + tn * 32 + frow]);
      }
    };
#pragma unroll
    for (int ks = 0; ks < kDepth; ++ks) rd(ks, ks);
    // one patch load every kEvery k-steps, all in the first half of the loop so that
    // the second half covers their latency
    constexpr int kEvery = D::NK / (2 * kLoads) > 1 ? D::NK / (2 * kLoads) : 1;
#pragma unroll
    for (int ks = 0; ks < D::NK; ++ks) {
      const int s = ks % (kDepth + 1);
      if (ks + kDepth < D::NK) rd(ks + kDepth, (ks + kDepth) % (kDepth + 1));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[s][tn], xf[s][tm], acc[tn][tm], 0, 0, 0);
        // a patch load between two pairs of MFMAs, which run while it issues
        if (tn == 0 && ks % kEvery == 0 && ks / kEvery < kLoads) {
          __builtin_amdgcn_sched_barrier(0);
          if (more) load_one(gn, b ^ 1, ks / kEvery);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // This wave's loads of the next patch have landed, and every wave is done with this
    // patch: the next iteration may compute from the other buffer and refill this one.
    d3_wait_vmcnt<0>();
    __syncthreads();

    // Epilogue from the accumulators: lane (frow, fk) holds, for block (tn, tm),
    // channels tn * 32 + 8q + 4fk + j (q, j in 0..3) of its pixel.
    const TileGeo g = tile_geo(t, per_img, tw);
    if (CS == 64 && a.pool2) {
      // Fused 2x2 max-pool: the max of the lane's two rows, then of the two lanes
      // (DPP quad_perm [1,0,3,2]); the window's even lane stores the pooled pixel's 16
      // channels as 8-byte pieces.  With ReLU it is applied to each value first and the
      // max taken on the bit patterns (non-negative floats order as their bits): for
      // every non-NaN sum that is the max of the four values followed by ReLU.
      const bool ok = (pcol & 1) == 0 && g.oh0 + prow < a.Ho && g.ow0 + pcol < a.Wo;
      const unsigned ybase = (unsigned)((g.n * Hy + (g.oh0 >> 1) + 2 * wave) * Wy + (g.ow0 >> 1)) * (unsigned)a.ldy * 2u;
      const unsigned yo = ok ? ybase + (unsigned)ylane : yoob;
      auto fs = [&](int tn, int tm, int e) {
        return __builtin_fmaf(acc[tn][tm][e], (&sc[tn][e >> 2].x)[e & 3], (&sh[tn][e >> 2].x)[e & 3]);
      };
#pragma unroll
      for (int tn = 0; tn < 2; ++tn) {
        int r[16];
        if (a.relu) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            r[e] = max(max(__float_as_int(fs(tn, 0, e)), 0), max(__float_as_int(fs(tn, 1, e)), 0));
            r[e] = max(r[e], __builtin_amdgcn_mov_dpp(r[e], 0xB1, 0xF, 0xF, true));
          }
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const float v = fmaxf(fs(tn, 0, e), fs(tn, 1, e));
            r[e] = __float_as_int(fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true))));
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const d3_u32x2 w = {d3_pack2(__int_as_float(r[4 * q]), __int_as_float(r[4 * q + 1])),
                              d3_pack2(__int_as_float(r[4 * q + 2]), __int_as_float(r[4 * q + 3]))};
          __builtin_amdgcn_raw_buffer_store_b64(w, yr, (int)(yo + tn * 64 + q * 16), 0, 0);
        }
      }
      continue;
    }
    // Without pool the wave's 64 rounded pixels go to an LDS region as [pixel][8 chunks]
    // (chunk c in slot c ^ swz(pixel)), then out with 16-byte stores of whole 128-byte
    // pixel rows, 8 lanes per pixel.  The region is the wave's share of the patch buffer
    // this tile was computed from (free until the next tile refills it), or with 8 input
    // channels a region of its own.
    uint4* stg = lds + (CS == 8 ? D::STG : pbase) + wave * 64 * 8;
    auto stage = [&](auto relu) {
#pragma unroll
      for (int tn = 0; tn < 2; ++tn)
#pragma unroll
        for (int tm = 0; tm < 2; ++tm)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              v[j] = __builtin_fmaf(acc[tn][tm][4 * q + j], (&sc[tn][q].x)[j], (&sh[tn][q].x)[j]);
              if constexpr (decltype(relu)::value) v[j] = d3_relu(v[j]);
            }
            const int p = tm * 32 + frow, c = tn * 4 + q;
            *(uint2*)((char*)(stg + p * 8 + (c ^ d3_swz(p))) + 8 * fk) = make_uint2(d3_pack2(v[0], v[1]), d3_pack2(v[2], v[3]));
          }
    };
    if (a.relu) stage(std::true_type{});
    else stage(std::false_type{});
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): the wave's staging writes have landed
    __builtin_amdgcn_wave_barrier();
    const int hlim = a.Ho - g.oh0 - 4 * wave, wlim = a.Wo - g.ow0 - (lane >> 3);
    const unsigned ybase = (unsigned)((g.n * a.Ho + g.oh0 + 4 * wave) * a.Wo + g.ow0) * (unsigned)a.ldy * 2u + (unsigned)ylane;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int p = r * 8 + (lane >> 3), c = lane & 7;
      const uint4 val = stg[p * 8 + (c ^ d3_swz(p))];
      const int dh = 2 * ((r & 3) >> 1) + (r >> 2), dw = 8 * (r & 1);   // step r's row and column in the wave's rows
      const bool ok = dh < hlim && dw < wlim;
      const unsigned yo = ok ? ybase + (unsigned)((dh * a.Wo + dw) * a.ldy * 2) : yoob;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(d3_u32x4, val), yr, (int)yo, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);   // reads done before the region is rewritten
    if constexpr (CS == 64) __syncthreads();   // every wave is done before the next tile refills the buffer
    else __builtin_amdgcn_wave_barrier();
  }
}

// Which instance takes this launch: 1 = 64 channels 3x3 (64 or, as two halves, 128
// output channels), 2 = 8 channels 3x3, 3 = 8 channels 7x7 stride 2; 0 = none.  The 8-channel instances ask for ReLU (a tap past
// the last adds exact zeros on either path, which can differ only in the sign of a zero
// sum, and ReLU maps both zeros to +0) and no fused pool (their epilogue stores whole
// pixels).
int conv_direct_variant(const ConvArgs& a) {
  if (a.res != nullptr || a.out_f32 || a.tap_stride != 0 || a.maxslot != nullptr || a.n_members > 1 ||
      (a.Nc != 64 && !(a.Nc == 128 && a.Cs == 64)) || a.Co_pad < a.Nc || a.c_write != a.Nc || a.ldy < a.Nc ||
      a.ldy % 4 != 0 || a.N < 1 ||
      a.kh != a.kw || (a.pool2 && (a.Ho % 2 != 0 || a.Wo % 2 != 0)))
    return 0;
  auto out_ok = [&](int k, int st) {
    const int pad = k / 2;
    return a.pad == pad && a.stride == st && a.Ho == (a.H + 2 * pad - k) / st + 1 &&
           a.Wo == (a.W + 2 * pad - k) / st + 1;
  };
  // outputs are addressed with 32-bit byte offsets (plus at most 112 bytes of immediate)
  const unsigned long long ybytes =
      (unsigned long long)a.N * (a.pool2 ? (a.Ho / 2) * (a.Wo / 2) : a.Ho * a.Wo) * a.ldy * 2;
  if (ybytes > 0xFFFFFF00ull) return 0;
  if (a.kh == 3 && a.Cs == 64 && a.K == 576 && a.Kp == 576 && out_ok(3, 1)) return 1;
  if (a.kh == 3 && a.Cs == 8 && a.K == 72 && a.Kp >= 80 && a.relu && !a.pool2 && out_ok(3, 1)) return 2;
  if (a.kh == 7 && a.Cs == 8 && a.K == 392 && a.Kp >= 400 && a.relu && !a.pool2 && out_ok(7, 2)) return 3;
  return 0;
}

bool conv_direct_fits(const ConvArgs& a) { return conv_direct_variant(a) != 0; }

hipError_t launch_conv_direct(const ConvArgs& a, hipStream_t s) {
  const int variant = conv_direct_variant(a);
  if (!variant) return hipErrorInvalidValue;
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
  const long long tiles = (long long)a.N * ((a.Ho + kTile - 1) / kTile) * ((a.Wo + kTile - 1) / kTile);
  const int per_cu = variant == 2 ? 2 : 1;   // workgroups that fit on a compute unit
  const int halves = a.Nc / 64;               // 128 output channels: two workgroups per tile
  const int grid = halves * (int)std::min<long long>(tiles, (long long)n_cu * per_cu / halves);
  if (variant == 1) launch((conv_direct_kernel<64, 3, 1, 1>), dim3(grid), dim3(256), s, a);
  else if (variant == 2) launch((conv_direct_kernel<8, 3, 1, 2>), dim3(grid), dim3(256), s, a);
  else launch((conv_direct_kernel<8, 7, 2, 1>), dim3(grid), dim3(256), s, a);
  return hipGetLastError();
}

template __global__ void conv_direct_kernel<64, 3, 1, 1>(ConvArgs);
template __global__ void conv_direct_kernel<8, 3, 1, 2>(ConvArgs);
template __global__ void conv_direct_kernel<8, 7, 2, 1>(ConvArgs);

}  // namespace rafiki
