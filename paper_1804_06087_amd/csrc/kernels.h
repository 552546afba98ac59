// Internal interface between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <hip/hip_ext.h>

namespace rafiki {

// Events the next kernel launch of this thread records at its own start and end (both
// null: untimed).  Set by the runtime's per-launch tracing; the dispatch itself records
// them, so the interval is the kernel's execution, not the queue around it.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

// Every kernel of the library is launched through this, so tracing can time it.  An
// untimed launch is a plain launch, which stream capture records into a graph.
template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  const LaunchEvents& ev = launch_events();
  if (ev.start || ev.stop)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev.start, ev.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

typedef uint16_t bf16_t;   // bfloat16 storage (upper half of an IEEE float)

// Grouped launches: models with identical layer lists run each layer as one launch,
// member k (up to kMaxGroup) on grid z = k with its own pointers; everything else
// (shapes, tile, splits) is shared, so every member's outputs are those of its own
// launch, bit for bit.
constexpr int kMaxGroup = 4;
struct GroupMember {
  const void* x;
  const void* w;
  const float* scale;
  const float* shift;
  const void* res;
  void* y;
  float* partial;
  unsigned* maxslot;
};
// Per-member input / output of the memory-bound kernels (n = 1: one tensor).
struct GroupIO {
  const void* x[kMaxGroup];
  void* y[kMaxGroup];
  unsigned* slot[kMaxGroup];
  int n;
};
inline GroupIO single_io(const void* x, void* y, unsigned* slot = nullptr) {
  GroupIO io{};
  io.x[0] = x;
  io.y[0] = y;
  io.slot[0] = slot;
  io.n = 1;
  return io;
}

// Implicit-GEMM convolution (also FC = 1x1 conv on a 1x1 image).
//   out[m, co] = epilogue( sum_k X[m, k] * Wp[co, k] )
//   m = (n, ho, wo) output pixel, k = (u, v, ci) kernel tap and input channel,
//   X[m, k] = x[n, ho*S - P + u, wo*S - P + v, ci] (zero outside the image).
// Epilogue: y = acc * scale[co] + shift[co] (+ res[m, co]), then ReLU if requested.
struct ConvArgs {
  const void* x;        // NHWC activations [N][H][W][Cs] (bf16 or fp32)
  const void* w;        // packed weights [Co_pad][Kp], K ordered (u, v, ci), zero padded
  const float* scale;   // [Co_pad] folded batch-norm scale (0 on padded channels)
  const float* shift;   // [Co_pad] folded shift incl. bias (0 on padded channels)
  const void* res;      // residual [M][ldy] (same type as x) or nullptr
  void* y;              // output [M][ldy], bf16/fp32 activations or fp32 logits
  float* partial;       // split-K partial sums [splits][M][Co_pad]
  int N, H, W, Cs;      // input geometry; Cs = storage channels (multiple of 8)
  int Ho, Wo, kh, kw, stride, pad;
  int M, K, Kp, Co_pad; // M = N*Ho*Wo; K = kh*kw*Cs; Kp = K rounded up to the K tile
  int Nc;               // output channels computed (tiles cover ceil(Nc / BN) * BN <= Co_pad rows)
  int c_write;          // channels written per row (<= Co_pad)
  int ldy;              // row stride of y and res, in elements
  int relu;
  int pool2;            // fused 2x2 stride-2 max-pool: GEMM row m is conv pixel (window m / 4, position
                        // m % 4 in row-major order within the window); y holds the pooled rows m / 4
  int out_f32;          // y is fp32 (bf16 kernels); fp32 kernels always write fp32
  int kt_per_split;     // K tiles per split (splits = gridDim.y)
  int n_tiles;          // channel tiles per row of the output tile grid
  // direct-to-LDS kernel: buffer sizes (bytes, < 2^31) and K decoding
  int x_bytes, w_bytes;
  int Cs8, K8;          // Cs / 8, K / 8
  unsigned mag_cs8;     // floor(x / Cs8) = umulhi(x, mag_cs8) (0 when Cs8 == 1)
  unsigned mag_kw;      // floor(x / kw)  = umulhi(x, mag_kw)  (0 when kw == 1)
  // Fused conv1d branches (aligned K order only; 0: off): every weight row is packed
  // over tap_stride taps per 64-channel block, but the rows of 64-row block b use only
  // their first taps_by_block[b] taps.  A tile runs the largest count over its rows and
  // skips the K tiles of the other taps, whose weights are all zero.
  int tap_stride;
  unsigned char taps_by_block[16];
  // With tap_stride > 0 and at most kMaxGatherTaps taps: gather the conv1d input rows
  // through token ids instead of reading a stored sequence.  Row (n, pos) of the input
  // is row tok[n * W + pos] of x, the embedding table [x_bytes / (2 Cs)][Cs]; ids
  // outside the table read zeros.  nullptr: x is the sequence itself.
  const int32_t* tok;
  // With tap_stride > 0, branches on 64-row blocks, Wo >= 128 and no split: the max
  // over positions is taken in the epilogue.  Each output row block b keeps positions
  // wo < W - taps_by_block[b] + 1; the bf16-rounded, ReLU'd values are max-reduced per
  // (request, channel) and merged with atomic max into maxslot [N][ldslot] as
  // order-preserving keys (max_key()), which start at 0.  nullptr: rows are stored.
  unsigned* maxslot;
  int ldslot;
  // Grouped launch: n_members > 1 replaces x, w, scale, shift, res, y, partial and
  // maxslot with members[blockIdx.z]'s (0 or 1: the fields above).
  int n_members;
  GroupMember members[kMaxGroup];
};
// The pointers of this workgroup's member of a grouped launch.  The members are
// picked with constant indices only: an index computed at run time into the argument
// struct would make the compiler copy the whole struct to scratch memory.
__device__ __forceinline__ void use_member(ConvArgs& a) {
  if (a.n_members > 1) {
    const unsigned z = blockIdx.z;
#pragma unroll
    for (int k = 1; k < kMaxGroup; ++k) {
      if (z == (unsigned)k) {
        a.x = a.members[k].x;
        a.w = a.members[k].w;
        a.scale = a.members[k].scale;
        a.shift = a.members[k].shift;
        a.res = a.members[k].res;
        a.y = a.members[k].y;
        a.partial = a.members[k].partial;
        a.maxslot = a.members[k].maxslot;
      }
    }
    if (z == 0) {
      a.x = a.members[0].x;
      a.w = a.members[0].w;
      a.scale = a.members[0].scale;
      a.shift = a.members[0].shift;
      a.res = a.members[0].res;
      a.y = a.members[0].y;
      a.partial = a.members[0].partial;
      a.maxslot = a.members[0].maxslot;
    }
  }
}
constexpr int kMaxGatherTaps = 8;
// Order-preserving key of a float for unsigned atomic max (0 is below every key).
__device__ __forceinline__ unsigned max_key(float f) {
  const unsigned u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float max_key_value(unsigned k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Direct-to-LDS pipelined bf16 MFMA kernel; cfg selects the tile configuration
// (kMfmaConfigs).  splits > 1 writes partial sums; finish with splitk_reduce.
struct MfmaConfig { int bm, bn, waves, stages, bk; };
constexpr int kNumMfmaConfigs = 43;
extern const MfmaConfig kMfmaConfigs[kNumMfmaConfigs];
hipError_t launch_conv_mfma(const ConvArgs& a, int cfg, int splits, hipStream_t s);
// Direct convolution of bf16 layers with 64 output channels (conv_direct.hip): the tuner's
// candidate kCfgDirect beside the GEMM tiles, bitwise equal to them.
constexpr int kCfgDirect = kNumMfmaConfigs;
bool conv_direct_fits(const ConvArgs& a);
hipError_t launch_conv_direct(const ConvArgs& a, hipStream_t s);
hipError_t launch_splitk_reduce(const ConvArgs& a, int splits, int in_bf16, hipStream_t s);
// fp32 direct kernel (CUDA-core style FMA loops; used by the fp32 precision mode).
hipError_t launch_conv_f32(const ConvArgs& a, hipStream_t s);

// NCHW fp32 images -> NHWC with Cs >= C storage channels (zero filled), bf16 or fp32.
hipError_t launch_stage_images(const float* x, void* y, int N, int C, int H, int W, int Cs, int to_bf16,
                               hipStream_t s);
// Max-pool k x k / stride / pad over NHWC (Cs channels).
hipError_t launch_maxpool(const GroupIO& io, int N, int H, int W, int Cs, int Ho, int Wo, int k, int stride, int pad,
                          int bf16, hipStream_t s);
inline hipError_t launch_maxpool(const void* x, void* y, int N, int H, int W, int Cs, int Ho, int Wo, int k,
                                 int stride, int pad, int bf16, hipStream_t s) {
  return launch_maxpool(single_io(x, y), N, H, W, Cs, Ho, Wo, k, stride, pad, bf16, s);
}
// Branches of a fused conv1d in the max/mean over positions: branch i occupies input
// channels [src[i], src[i] + cnt[i]), reduces them over its first len[i] positions and
// writes output channels [dst[i], dst[i] + cnt[i]) of rows ldy wide; output channels
// zero_from .. ldy - 1 are set to zero; input channels in no branch are not written.
// n = 0: every channel over all positions, the output laid out as the input.
constexpr int kMaxReduceSegs = 8;
struct ReduceSegs {
  int n, ldy, zero_from;
  int src[kMaxReduceSegs], dst[kMaxReduceSegs], cnt[kMaxReduceSegs], len[kMaxReduceSegs];
};
// Global average pool NHWC [N][HW][Cs] -> [N][Cs]; also max over time when is_max.
hipError_t launch_spatial_reduce(const GroupIO& io, int N, int HW, int Cs, int is_max, int bf16, hipStream_t s,
                                 const ReduceSegs* segs = nullptr);
inline hipError_t launch_spatial_reduce(const void* x, void* y, int N, int HW, int Cs, int is_max, int bf16,
                                        hipStream_t s, const ReduceSegs* segs = nullptr) {
  return launch_spatial_reduce(single_io(x, y), N, HW, Cs, is_max, bf16, s, segs);
}
// Fused branches' max in the GEMM epilogue: y[n][dst_i + k] = bf16 of slot row n at
// channel src_i + k for each branch, zeros from zero_from to ldy; every slot read is
// reset to 0 for the next call.
hipError_t launch_maxslot_finish(const GroupIO& io, int ldslot, int N, const ReduceSegs& sg, hipStream_t s);
inline hipError_t launch_maxslot_finish(unsigned* slot, int ldslot, void* y, int N, const ReduceSegs& sg,
                                        hipStream_t s) {
  return launch_maxslot_finish(single_io(nullptr, y, slot), ldslot, N, sg, s);
}
// Embedding gather: tokens [N][L] -> y [N][L][Cs] rows of table [vocab][Cs]; ids
// outside [0, vocab) give zero rows.
hipError_t launch_embed_gather(const int32_t* tok, const void* table, void* y, int N, int L, int Cs, int vocab,
                               int bf16, hipStream_t s);
// Concatenate vectors: y[b, 0:c1] = a[b, 0:c1], y[b, c1:c1+c2] = b[b, 0:c2], zero after.
hipError_t launch_concat(const void* a, int ca, int lda, const void* b, int cb, int ldb, void* y, int ldy,
                         int N, int bf16, hipStream_t s);

// Ensemble combine over S selected models' fp32 logits.
struct CombineArgs {
  const float* logits;  // base of [n_models][ld_model] slots; model m at logits + m * ld_model
  long long ld_model;   // elements between consecutive model slots
  int sel[32];          // selected model indices
  int S;                // number of selected models (>= 1)
  int n, C;
  float* probs;         // [n][C]
  int32_t* labels;      // [n]
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);
// Majority vote over the same slots: probs <- vote fractions, labels <- winner.
hipError_t launch_vote(const CombineArgs& a, hipStream_t s);

// Whole-network kernel for small image CNNs (fused_net.hip): one workgroup of
// kFusedWaves waves runs one model's layer program on one image, the activations in
// an LDS arena of kFusedLdsBytes (tensors [pixel][Cs] bf16, 8 <= Cs <= 64 a power of
// two, in a swizzled chunk order), followed in LDS by 128 zero bytes and the model's
// folded scale / shift table of at most kFusedTableBytes.
constexpr int kFusedWaves = 4;
constexpr int kFusedLdsBytes = 64 * 1024;
constexpr int kFusedTableBytes = 8 * 1024;
constexpr int kFusedMaxLayers = 64;
// F_INPUT copies the staged image [Ho * Wo][Cso] to out_off and the scale / shift
// table (`scale`, c_write bytes) to ss_off; F_END ends a program.
enum FusedOpKind { F_END = 0, F_INPUT = 1, F_CONV = 2, F_GAP = 3, F_FC = 4 };
struct FusedLayer {
  int op;                        // FusedOpKind
  int in_off, res_off, out_off;  // LDS byte offsets of the input, residual (-1: none) and output
  int H, W, Cs;                  // input geometry, storage channels
  int Ho, Wo, Cso;               // output geometry; Cso = output row stride (FC: logits row length)
  int c_write;                   // output channels written
  int kh, kw, stride, pad, relu;
  int K, Kp;                     // K = kh * kw * Cs terms, packed weight row length
  int n_cb, n_pb, ch;            // 32-channel blocks, 32-pixel blocks, pixel blocks per wave task
  int lwo;                       // log2(Wo)
  int ss_off;                    // LDS offset of this layer's scale [c4] then shift [c4], c4 = c_write rounded to 4
  int tmp_off;                   // GAP: LDS scratch of the partial sums
  const bf16_t* w;               // weights in fragment order [n_cb][ceil(K / 16)][64 lanes][8]: lane
                                 // fk * 32 + r holds row cb * 32 + r, terms 16 g + 8 fk .. + 7, K in
                                 // (tap, channel) order
  const float* scale;            // F_INPUT: the model's scale / shift table in global memory
};
struct FusedNetArgs {
  const FusedLayer* progs;   // [n_models][kFusedMaxLayers] programs, each ended by F_END
  float* logits;             // model m's logits at logits + m * ld_model, rows of the FC's Cso
  long long ld_model;
  unsigned mask;             // selected models; grid y = the y-th set bit
  const bf16_t* in;          // staged images [n][Ho * Wo][Cso] of the programs' F_INPUT
};
hipError_t launch_fused_net(const FusedNetArgs& a, int n, int n_models, hipStream_t s);

// Peak probes: register-resident bf16 MFMA loop (out [blocks * 4] checksums) and a
// streaming 16-byte read of words16 words (out [blocks * 4]).
hipError_t launch_probe_mfma(int blocks, int iters, float* out, hipStream_t s);
hipError_t launch_probe_read(const void* x, long long words16, int blocks, unsigned* out, hipStream_t s);
hipError_t launch_probe_mainloop(int variant, bool sync, int blocks, int ktiles, float* out, hipStream_t s);

}  // namespace rafiki
