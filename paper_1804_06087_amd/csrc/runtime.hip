// Host runtime and C ABI of the ensemble-inference library.
//
// create: validate the layer lists, infer tensor shapes, fold batch-norm into a
//   per-channel fp32 (scale, shift) computed in fp64, round weights to the compute
//   precision, pack them in the kernels' [Co_pad][Kp] (u, v, ci) order, upload, and
//   plan each model's activation workspace by liveness for max_batch requests.
// infer: stage the request batch once (NCHW fp32 -> NHWC) on the caller's stream, run
//   the forward pass of every selected model into its logits slot (on the models' own
//   streams, in the schedule timed for this batch size and subset, or replayed as a
//   graph), join back on the caller's stream, then combine.  The first call with a
//   new batch size also times every GEMM op's tile candidates inside forward passes.
#include "rafiki_ensemble.h"
#include "kernels.h"
#include "greedy.h"

#include <algorithm>
#include <chrono>
#include <climits>
#include <cmath>
#include <cstring>
#include <cstdlib>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

using namespace rafiki;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }
inline size_t round_up_sz(size_t x, size_t m) { return (x + m - 1) / m * m; }

// Host float -> bf16 bits, nearest with ties to even (finite values).
inline uint16_t host_f2bf(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

enum TKind { T_IMG = 0, T_VEC = 1, T_SEQ = 2, T_TOK = 3 };

struct Tensor {
  int kind = T_IMG;
  int c = 0, h = 1, w = 1, Cs = 0;   // logical channels, spatial size, storage channels
  size_t off = 0;                    // byte offset in the model arena
  int last_use = -1;
  bool is_logits = false;
  size_t item_elems() const { return (size_t)h * w * Cs; }
};

enum OpKind { O_CONV = 0, O_MAXPOOL, O_GAP, O_EMBED, O_CONV1D, O_CONCAT };

struct Op {
  int kind = O_CONV;
  int in = -1, in2 = -1, out = -1;
  // GEMM-like ops (conv2d, FC, conv1d)
  int H = 1, W = 1, Cs_in = 0, Ho = 1, Wo = 1, kh = 1, kw = 1, stride = 1, pad = 0, relu = 0;
  int K = 0, Kp = 0, Co_pad = 0, c_out = 0;
  int cin_l = 0;        // logical input channels (algorithmic FLOP / byte counts)
  void* d_w = nullptr;
  float* d_scale = nullptr;
  float* d_shift = nullptr;
  // pooling
  int k = 1;
  // conv2d: a 2x2 stride-2 max-pool fused into the epilogue; `out` is the pooled tensor
  int pool2 = 0;
  // conv1d: pre-max scratch [n][T][Cs_out] in the arena
  size_t tmp_off = 0;
  // conv1d running several fused branches (nseg > 0): branch i owns output channels
  // [seg_end[i - 1], seg_end[i]), GEMM rows from seg_row[i] on, and has a kernel of
  // seg_kw[i] taps; tap_stride / taps_by_block as in ConvArgs
  int nseg = 0;
  int seg_end[kMaxReduceSegs] = {}, seg_kw[kMaxReduceSegs] = {}, seg_row[kMaxReduceSegs] = {};
  int tap_stride = 0;
  unsigned char taps_by_block[16] = {};
  // fused branches reading the token ids: input rows gathered from this table
  const void* table = nullptr;
  // fused branches whose max is taken in the GEMM epilogue (unsplit launches): atomic
  // max keys [max_batch][ldslot], zero between calls
  unsigned* d_slot = nullptr;
  int ldslot = 0;
  // concat
  int ca = 0, cb = 0;
};

struct Model {
  std::vector<Op> ops;
  std::vector<Tensor> tensors;
  char* d_arena = nullptr;
  size_t arena_bytes = 0;
  float* d_partial = nullptr;     // split-K partial sums (per model: models may run concurrently)
  size_t partial_bytes = 0;
  hipStream_t stream = nullptr;   // the model's own stream for concurrent ensembles
  hipEvent_t done = nullptr;      // recorded on `stream` after the model's last kernel
  void* d_staged_own = nullptr;   // the model's own staged input (asynchronous serving)
  // Whole-network program (fused_net.hip) when every layer fits that kernel; empty if not.
  std::vector<FusedLayer> fprog;
};

struct FreeList {
  struct B { size_t off, size; };
  std::vector<B> free;
  size_t top = 0;
  size_t alloc(size_t n) {
    n = round_up_sz(std::max<size_t>(n, 1), 256);
    for (size_t i = 0; i < free.size(); ++i) {
      if (free[i].size >= n) {
        size_t off = free[i].off;
        free[i].off += n;
        free[i].size -= n;
        if (free[i].size == 0) free.erase(free.begin() + i);
        return off;
      }
    }
    size_t off = top;
    top += n;
    return off;
  }
  void release(size_t off, size_t n) {
    n = round_up_sz(std::max<size_t>(n, 1), 256);
    free.push_back({off, n});
    std::sort(free.begin(), free.end(), [](const B& a, const B& b) { return a.off < b.off; });
    std::vector<B> merged;
    for (auto& b : free) {
      if (!merged.empty() && merged.back().off + merged.back().size == b.off) merged.back().size += b.size;
      else merged.push_back(b);
    }
    free.swap(merged);
  }
};

}  // namespace

// Opt-in per-launch timing: HIP events recorded on the launch stream around each
// kernel, resolved by rafiki_ensemble_trace_read.
struct Tracer {
  bool on = false;
  bool concurrent = false;   // keep the models' own streams and schedule while tracing
  struct Rec { int kind, model, layer; double flops, bytes; hipEvent_t a, b; int tile_cfg, splits; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  hipEvent_t next() {
    if (used == pool.size()) {
      hipEvent_t ev = nullptr;
      if (hipEventCreate(&ev) != hipSuccess) return nullptr;
      pool.push_back(ev);
    }
    return pool[used++];
  }
  ~Tracer() {
    for (hipEvent_t ev : pool) (void)hipEventDestroy(ev);
  }
};

struct rafiki_ensemble_s {
  int n_models = 0, n_classes = 0, precision = 0, max_batch = 0;
  mutable Tracer trace;
  int input_kind = 0, C = 0, H = 0, W = 0, vocab = 0, in_Cs = 0;
  int device = 0;
  bool dry = false;   // validation pass: shapes only, no packing, no device calls
  std::vector<Model> models;
  void* d_staged = nullptr;
  float* d_logits = nullptr;
  hipEvent_t staged_ev = nullptr;   // recorded on the caller's stream after staging
  bool concurrent = true;           // run selected models on their own streams
  std::vector<void*> allocs;
  // Tuned tile configuration per batch size, model and op (-1: not a GEMM op).
  std::map<int, std::vector<std::vector<int>>> tuned;
  // The same per batch size, except that each unsplit GEMM layer with an output map of at
  // most 14 x 14 pixels takes its fastest lean tile (8 waves, at least 128 x 128, K tiles
  // of 64, at most 64 KB of LDS ring): more FLOPs per loaded byte than the small tiles those layers
  // prefer alone, and room on each compute unit for the other models' workgroups when
  // models run concurrently.  Every tile gives the same bits.
  std::map<int, std::vector<std::vector<int>>> tuned_lean;
  // tuned_lean with every direct-conv choice replaced by the layer's fastest GEMM tile:
  // the direct kernel's persistent workgroups fill each compute unit's LDS, which leaves
  // no room for the other lane's workgroups while it runs.
  std::map<int, std::vector<std::vector<int>>> tuned_lean_gemm;
  // Per batch size: each model's forward time alone, estimated when tuning (sum of the
  // chosen tiles' times; GEMM FLOPs / 1e12 when tiles are not timed).
  std::map<int, std::vector<double>> model_ms;
  // Per (batch size, subset): the schedule of the selected models' forward passes
  // chosen by timing (solo -1: all concurrent; solo m: model m alone on one lane, the
  // others one after another on a second lane, longest estimated alone time first, or
  // shortest first when `ascending`).
  // pa >= 0: models pa and pb run paired on one lane (their aligned ops as two-member
  // launches) and the other selected models one after another on a second lane; solo
  // and ascending are then unused.
  struct Sched {
    int solo = -1, ascending = 0, pa = -1, pb = -1;
    int lean = 0;   // 1: the small-map layers take their lean tiles (tuned_lean); 2: also the
                    // solo model's direct-conv layers take their fastest GEMM tile (tuned_lean_gemm)
  };
  std::map<std::pair<int, uint32_t>, Sched> schedule;
  // Pairable models (a < b) of different layer lists: the merged op order of the two,
  // each step (i, j) an op of a and an op of b with the same launch signature, or one of
  // them -1 (that model's op alone).
  std::map<std::pair<int, int>, std::vector<std::pair<int, int>>> pairing;
  bool tune_schedule = true;
  bool autotune = true;
  bool fuse_branches = true;        // fuse sibling max-over-time convolutions (bf16)
  bool lean_policy = true;          // the schedule timing also tries the lean tiles
  // Models with identical layer lists share a group id (the lowest index among them);
  // a selection within one group runs as grouped launches (RAFIKI_GROUPED=0: never).
  std::vector<int> group_of;
  bool grouped = true;
  int force_tile = -1;              // diagnostic override of the tuned configuration
  // Forward passes replayed as HIP graphs, one per (batch size, model subset): every
  // kernel argument inside them (weights, arenas, staged input, logits workspace,
  // tuned tiles) is fixed once the batch size has been tuned.  Staging and the combine,
  // which touch the caller's buffers, are launched outside the graph.
  struct GraphExec {
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
  };
  bool use_graphs = false;          // opt-in: replay measured no faster than the eager launches
  std::map<std::pair<int, uint32_t>, GraphExec> graphs;
  hipStream_t capture_stream = nullptr;
  void* d_tokens = nullptr;         // token ids copied here when a graph reads them
  long long graph_replays = 0, graph_failures = 0;
  // Device address of the library's static scratch array on this handle's device
  // (resolved at create; null with the reason in scratch_err if that failed).
  void* scratch = nullptr;
  std::string scratch_err;
  // Whole-network kernel: the models' programs [n_models][kFusedMaxLayers] on the
  // device (null if no model fits it); RAFIKI_FUSED_NET=0 at create turns it off.
  bool fused_net = true;
  FusedLayer* d_fprog = nullptr;
  size_t esz() const { return precision == RAFIKI_BF16 ? 2 : 4; }
  void drop_graphs() {
    for (auto& kv : graphs) {
      if (kv.second.exec) (void)hipGraphExecDestroy(kv.second.exec);
      if (kv.second.graph) (void)hipGraphDestroy(kv.second.graph);
    }
    graphs.clear();
  }
  ~rafiki_ensemble_s() {
    drop_graphs();
    if (capture_stream) (void)hipStreamDestroy(capture_stream);
    for (Model& M : models) {
      if (M.done) (void)hipEventDestroy(M.done);
      if (M.stream) (void)hipStreamDestroy(M.stream);
    }
    if (staged_ev) (void)hipEventDestroy(staged_ev);
    for (void* p : allocs) (void)hipFree(p);
  }
};

namespace {

int dev_alloc(rafiki_ensemble_s* e, void** p, size_t bytes) {
  *p = nullptr;
  if (e->dry) return RAFIKI_OK;
  if (bytes == 0) bytes = 256;
  hipError_t st = hipMalloc(p, bytes);
  if (st != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    return fail(st == hipErrorOutOfMemory ? RAFIKI_ERR_NOMEM : RAFIKI_ERR_HIP,
                std::string("hipMalloc of ") + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(st));
  }
  e->allocs.push_back(*p);
  return RAFIKI_OK;
}

int upload(rafiki_ensemble_s* e, void** dst, const void* src, size_t bytes) {
  int rc = dev_alloc(e, dst, bytes);
  if (rc || e->dry) return rc;
  hipError_t st = hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipMemcpy failed: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

// bf16 GEMM tiling.  Weight rows are padded to 256 so every tile configuration fits.
constexpr int kCoPadBf16 = 256;

// Configurations whose channel tile suits c_out (at most one partly used tile row).
bool cfg_fits(int cfg, int c_out) {
  if (cfg < 0 || cfg >= kNumMfmaConfigs) return false;
  const int bn = kMfmaConfigs[cfg].bn;
  if (c_out <= 32) return bn == 32;
  if (c_out <= 64) return bn <= 64;
  return bn <= round_up(c_out, 64) && bn >= 64;
}
// Split K when the output tile grid of the smallest tiles cannot fill the 256
// compute units.  Depends only on the GEMM shape, so results do not depend on tuning.
int choose_splits(int M, int c_out, int ktiles) {
  const int tiles = ((M + 63) / 64) * ((c_out + 127) / 128);
  if (tiles >= 256 || ktiles < 12) return 1;
  int s = std::min((512 + tiles - 1) / tiles, ktiles / 4);
  s = std::max(1, std::min(s, 64));
  const int per = (ktiles + s - 1) / s;
  return (ktiles + per - 1) / per;
}
// Untuned tile of split-K launches.
int split_cfg(int c_out) { return c_out <= 32 ? 10 : (c_out <= 64 ? 8 : 6); }
// Untuned default: the 64-pixel tiles are the most robust across shapes.
int default_cfg(int c_out) { return c_out <= 32 ? 10 : (c_out <= 64 ? 8 : 6); }

// Pack a GEMM-like weight into [Co_pad][Kp] over Cs_in storage channels.  K order:
// (channel block of 64, tap, channel) for the bf16 kernel's aligned path (bf16 and
// Cs_in % 64 == 0), else (tap, channel), the order the fp32 kernel reads.
// `src_index(co, ci, u, v)` gives the canonical flat index.
template <class F>
std::vector<float> pack_weight(bool bf16, int c_out, int c_in, int kh, int kw, int Cs_in, int Co_pad, int Kp,
                               F src_index, const float* w) {
  std::vector<float> out((size_t)Co_pad * Kp, 0.f);
  const bool aligned = bf16 && Cs_in % 64 == 0;
  const int taps = kh * kw;
  for (int co = 0; co < c_out; ++co)
    for (int u = 0; u < kh; ++u)
      for (int v = 0; v < kw; ++v)
        for (int ci = 0; ci < c_in; ++ci) {
          const int tap = u * kw + v;
          const size_t k = aligned ? ((size_t)(ci / 64) * taps + tap) * 64 + ci % 64 : (size_t)tap * Cs_in + ci;
          out[(size_t)co * Kp + k] = w[src_index(co, ci, u, v)];
        }
  return out;
}

int upload_weights(rafiki_ensemble_s* e, Op& op, const std::vector<float>& packed) {
  if (e->precision == RAFIKI_BF16) {
    std::vector<uint16_t> b(packed.size());
    for (size_t i = 0; i < packed.size(); ++i) b[i] = host_f2bf(packed[i]);
    return upload(e, &op.d_w, b.data(), b.size() * 2);
  }
  return upload(e, &op.d_w, packed.data(), packed.size() * 4);
}

// GEMM weights packed as [Co_pad][Kp]: uploaded as they are for the bf16 kernel, and
// transposed to [Kp][Co_pad] for the fp32 kernel, whose lanes read the weights of 4
// consecutive output channels of one K index as one 16-byte load.
int upload_gemm_weights(rafiki_ensemble_s* e, Op& op, const std::vector<float>& packed) {
  if (e->precision == RAFIKI_BF16) return upload_weights(e, op, packed);
  std::vector<float> t(packed.size());
  for (int co = 0; co < op.Co_pad; ++co)
    for (int k = 0; k < op.Kp; ++k) t[(size_t)k * op.Co_pad + co] = packed[(size_t)co * op.Kp + k];
  return upload_weights(e, op, t);
}

// Fold inference batch-norm and bias: y = s * conv + t, s = gamma / sqrt(var + eps),
// t = beta - mean * s + s * bias, evaluated in fp64 and rounded once to fp32.
void fold_into(const rafiki_layer& L, float* s, float* t) {
  const bool bn = L.bn_gamma != nullptr;
  for (int c = 0; c < L.c_out; ++c) {
    const double b = L.bias ? (double)L.bias[c] : 0.0;
    if (bn) {
      const double sc = (double)L.bn_gamma[c] / std::sqrt((double)L.bn_var[c] + (double)L.bn_eps);
      s[c] = (float)sc;
      t[c] = (float)((double)L.bn_beta[c] - (double)L.bn_mean[c] * sc + sc * b);
    } else {
      s[c] = 1.f;
      t[c] = (float)b;
    }
  }
}

int upload_fold(rafiki_ensemble_s* e, Op& op, const std::vector<float>& s, const std::vector<float>& t) {
  int rc = upload(e, (void**)&op.d_scale, s.data(), s.size() * 4);
  if (rc) return rc;
  return upload(e, (void**)&op.d_shift, t.data(), t.size() * 4);
}

int upload_fold(rafiki_ensemble_s* e, Op& op, const rafiki_layer& L) {
  std::vector<float> s(op.Co_pad, 0.f), t(op.Co_pad, 0.f);
  fold_into(L, s.data(), t.data());
  int rc = upload(e, (void**)&op.d_scale, s.data(), s.size() * 4);
  if (rc) return rc;
  return upload(e, (void**)&op.d_shift, t.data(), t.size() * 4);
}

// Storage channels of an activation: a multiple of 8 (one 16-byte chunk), or of 64 in
// bf16 when that pads by at most an eighth, so that the GEMMs reading it take the
// kernel's channel-block K order (300-dimensional embeddings: 320; the TextCNN
// convolutions then run 14 % faster).  Padded channels hold zeros.
int storage_channels(int c, bool bf16) {
  const int c64 = round_up(c, 64);
  return bf16 && c > 64 && 8 * c64 <= 9 * c ? c64 : round_up(c, 8);
}

std::string lname(int m, int i) { return "model " + std::to_string(m) + " layer " + std::to_string(i) + ": "; }

// Branches of a model that run as one GEMM: max-over-time convolutions reading one
// sequence whose outputs meet only in a tree of concatenations (the TextCNN's kernel
// widths 3, 4 and 5, joined in order).  The branches' filters become the rows of one
// weight matrix over the widest kernel's taps, a narrower branch's missing taps holding
// zero weights; past the end of the sequence the GEMM reads the hardware's zeros, so
// it can run over the positions of the narrowest branch.  Every output sums its own
// products in its own K order with only exact zero products added, so each value is
// bitwise that of its separate branch.  The max over time then reduces each branch's
// channels over that branch's W - kw + 1 positions and writes the concatenated vector
// directly: the concatenations disappear.
struct BranchGroup {
  int root = -1;                  // the outermost concatenation
  std::vector<int> branches;      // convolution layers, in channel order
  std::vector<int> concats;       // the concatenations inside the tree
};

void branch_leaves(const rafiki_model_desc& md, const std::vector<int>& readers, int t, BranchGroup& g, bool& ok) {
  const rafiki_layer& L = md.layers[t];
  for (int src : {L.input, L.input2}) {
    if (src < 0 || src >= t) {
      ok = false;
      return;
    }
    if (md.layers[src].op == RAFIKI_OP_CONCAT && readers[src] == 1) {
      g.concats.push_back(src);
      branch_leaves(md, readers, src, g, ok);
      if (!ok) return;
    } else {
      g.branches.push_back(src);
    }
  }
}

std::vector<BranchGroup> find_branch_groups(const rafiki_model_desc& md) {
  const int nl = md.n_layers;
  std::vector<int> readers(nl, 0), reader(nl, -1);
  for (int i = 0; i < nl; ++i)
    for (int src : {md.layers[i].input, md.layers[i].input2})
      if (src >= 0 && src < i) {
        ++readers[src];
        reader[src] = i;
      }
  std::vector<BranchGroup> groups;
  for (int r = 0; r < nl; ++r) {
    if (md.layers[r].op != RAFIKI_OP_CONCAT) continue;
    if (readers[r] == 1 && md.layers[reader[r]].op == RAFIKI_OP_CONCAT) continue;   // inside a larger tree
    BranchGroup g;
    g.root = r;
    bool ok = true;
    branch_leaves(md, readers, r, g, ok);
    if (!ok || g.branches.size() < 2 || g.branches.size() > (size_t)kMaxReduceSegs) continue;
    const rafiki_layer& b0 = md.layers[g.branches[0]];
    for (int b : g.branches) {
      const rafiki_layer& L = md.layers[b];
      ok = ok && L.op == RAFIKI_OP_CONV1D_MAXTIME && readers[b] == 1 && L.input == b0.input &&
           L.c_in == b0.c_in && (L.relu != 0) == (b0.relu != 0) && L.weight && L.kw >= 1;
    }
    if (ok) groups.push_back(std::move(g));
  }
  return groups;
}

// Replace each group's branch convolutions and concatenations by one conv1d op that
// writes the group's root tensor; packs and uploads its weights and folded scale and
// shift unless the handle is in its validation pass.
int fuse_branches(rafiki_ensemble_s* e, const rafiki_model_desc& md, Model& M, const std::vector<BranchGroup>& groups) {
  std::vector<int> group_of(M.ops.size(), -1);
  std::vector<Op> fused(groups.size());
  for (size_t gi = 0; gi < groups.size(); ++gi) {
    const BranchGroup& g = groups[gi];
    group_of[g.root] = (int)gi;
    for (int t : g.branches) group_of[t] = (int)gi;
    for (int t : g.concats) group_of[t] = (int)gi;
    Op m = M.ops[g.branches[0]];
    m.out = g.root;
    m.nseg = (int)g.branches.size();
    int kw_max = 0, kw_min = 1 << 30, c = 0, rows_dense = 0, rows_64 = 0;
    for (int i = 0; i < m.nseg; ++i) {
      const Op& b = M.ops[g.branches[i]];
      kw_max = std::max(kw_max, b.kw);
      kw_min = std::min(kw_min, b.kw);
      c += b.c_out;
      m.seg_end[i] = c;
      m.seg_kw[i] = b.kw;
      rows_dense += b.c_out;
      rows_64 = round_up(rows_64, 64) + b.c_out;
    }
    if (c != M.tensors[g.root].c) return fail(RAFIKI_ERR_INVALID, "internal: fused branch channels");
    // With the aligned K order a tile skips the taps its rows lack; branches start on
    // 64-row blocks when that adds at most a third to the GEMM's rows, so that tiles
    // seldom mix kernel widths.
    const bool aligned = m.Cs_in % 64 == 0;
    const bool pad64 = aligned && 3 * rows_64 <= 4 * rows_dense && round_up(rows_64, 64) <= 16 * 64;
    int rows = 0;
    for (int i = 0; i < m.nseg; ++i) {
      if (pad64) rows = round_up(rows, 64);
      m.seg_row[i] = rows;
      rows += m.seg_end[i] - (i ? m.seg_end[i - 1] : 0);
    }
    m.kw = kw_max; m.Wo = m.W - kw_min + 1; m.c_out = rows;
    m.K = kw_max * m.Cs_in;
    m.Co_pad = round_up(rows, kCoPadBf16);
    m.Kp = round_up(m.K, 64);
    m.tap_stride = 0;
    if (aligned && round_up(rows, 64) <= 16 * 64) {
      m.tap_stride = kw_max;
      for (int b = 0; b < 16; ++b) {
        int t = 1;
        for (int i = 0; i < m.nseg; ++i) {
          const int r0 = m.seg_row[i], r1 = r0 + m.seg_end[i] - (i ? m.seg_end[i - 1] : 0);
          if (r0 < 64 * (b + 1) && r1 > 64 * b) t = std::max(t, m.seg_kw[i]);
        }
        m.taps_by_block[b] = (unsigned char)t;
      }
    }
    m.d_w = nullptr; m.d_scale = nullptr; m.d_shift = nullptr;
    if (!e->dry) {
      // K order as pack_weight's over kw_max taps: (channel block of 64, tap, channel)
      // when aligned, else (tap, channel)
      std::vector<float> packed((size_t)m.Co_pad * m.Kp, 0.f), sc(m.Co_pad, 0.f), sh(m.Co_pad, 0.f);
      for (int i = 0; i < m.nseg; ++i) {
        const rafiki_layer& L = md.layers[g.branches[i]];
        const int cin = L.c_in, kw = L.kw, o = m.seg_row[i];
        for (int co = 0; co < L.c_out; ++co)
          for (int v = 0; v < kw; ++v)
            for (int ci = 0; ci < cin; ++ci) {
              const size_t k = aligned ? ((size_t)(ci / 64) * kw_max + v) * 64 + ci % 64 : (size_t)v * m.Cs_in + ci;
              packed[(size_t)(o + co) * m.Kp + k] = L.weight[((size_t)co * cin + ci) * kw + v];
            }
        fold_into(L, sc.data() + o, sh.data() + o);
      }
      int rc = upload_weights(e, m, packed);
      if (!rc) rc = upload_fold(e, m, sc, sh);
      if (rc) return rc;
    }
    // Branches on their own 64-row blocks and requests of at least 128 positions (a
    // wave tile then spans at most two requests): the max can be taken in the GEMM
    // epilogue, into slots that start at zero and are reset as they are read.
    if (pad64 && m.tap_stride > 0 && m.Wo >= 128) {
      m.ldslot = round_up(rows, 8);
      const size_t bytes = (size_t)e->max_batch * m.ldslot * 4;
      int rc = dev_alloc(e, (void**)&m.d_slot, bytes);
      if (rc) return rc;
      if (!e->dry) {
        const hipError_t st = hipMemset(m.d_slot, 0, bytes);
        if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipMemset: ") + hipGetErrorString(st));
      }
    }
    fused[gi] = m;
  }
  std::vector<Op> ops;
  for (const Op& op : M.ops) {
    const int gi = op.out >= 0 && op.out < (int)group_of.size() ? group_of[op.out] : -1;
    if (gi < 0) ops.push_back(op);
    else if (op.out == groups[gi].root) ops.push_back(fused[gi]);
  }
  M.ops.swap(ops);
  return RAFIKI_OK;
}

// Validate one model, infer shapes, build its ops and upload its parameters.
int build_model(rafiki_ensemble_s* e, int mi, const rafiki_model_desc& md, Model& M) {
  if (md.n_layers < 1 || !md.layers) return fail(RAFIKI_ERR_INVALID, "model " + std::to_string(mi) + ": no layers");
  if (md.n_classes < 1) return fail(RAFIKI_ERR_INVALID, "model " + std::to_string(mi) + ": n_classes < 1");
  Tensor in;
  if (e->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32) {
    in.kind = T_IMG; in.c = e->C; in.h = e->H; in.w = e->W; in.Cs = e->in_Cs;
  } else {
    in.kind = T_TOK; in.c = 1; in.h = 1; in.w = e->H; in.Cs = 1;
  }
  const bool bf = e->precision == RAFIKI_BF16;
  auto tin = [&](int id) -> const Tensor& { return id < 0 ? in : M.tensors[id]; };
  M.tensors.resize(md.n_layers);
  const std::vector<BranchGroup> groups =
      bf && e->fuse_branches ? find_branch_groups(md) : std::vector<BranchGroup>();
  std::vector<char> in_group(md.n_layers, 0);
  for (const BranchGroup& g : groups)
    for (int b : g.branches) in_group[b] = 1;
  for (int i = 0; i < md.n_layers; ++i) {
    const rafiki_layer& L = md.layers[i];
    const std::string ln = lname(mi, i);
    if (L.input < -1 || L.input >= i) return fail(RAFIKI_ERR_INVALID, ln + "input id out of range");
    if (L.input2 < -1 || L.input2 >= i) return fail(RAFIKI_ERR_INVALID, ln + "input2 id out of range");
    const Tensor& x = tin(L.input);
    Tensor& y = M.tensors[i];
    Op op;
    op.in = L.input; op.in2 = L.input2; op.out = i; op.relu = L.relu ? 1 : 0;
    const bool has_bn = L.bn_gamma || L.bn_beta || L.bn_mean || L.bn_var;
    if (has_bn && !(L.bn_gamma && L.bn_beta && L.bn_mean && L.bn_var))
      return fail(RAFIKI_ERR_INVALID, ln + "batch-norm needs all of gamma, beta, mean, var");
    if (has_bn && !(L.bn_eps >= 0.f)) return fail(RAFIKI_ERR_INVALID, ln + "bn_eps must be >= 0");
    switch (L.op) {
      case RAFIKI_OP_CONV2D: {
        if (x.kind != T_IMG) return fail(RAFIKI_ERR_INVALID, ln + "conv2d needs an image tensor");
        if (L.c_in != x.c || L.c_out < 1) return fail(RAFIKI_ERR_INVALID, ln + "conv2d channel mismatch");
        if (L.kh < 1 || L.kw < 1 || L.stride < 1 || L.pad < 0 || !L.weight)
          return fail(RAFIKI_ERR_INVALID, ln + "conv2d geometry or weight invalid");
        const int Ho = (x.h + 2 * L.pad - L.kh) / L.stride + 1, Wo = (x.w + 2 * L.pad - L.kw) / L.stride + 1;
        if (x.h + 2 * L.pad < L.kh || x.w + 2 * L.pad < L.kw || Ho < 1 || Wo < 1)
          return fail(RAFIKI_ERR_INVALID, ln + "conv2d output would be empty");
        y.kind = T_IMG; y.c = L.c_out; y.h = Ho; y.w = Wo; y.Cs = storage_channels(L.c_out, bf);
        if (L.input2 >= 0) {
          const Tensor& r = M.tensors[L.input2];
          if (r.kind != T_IMG || r.c != y.c || r.h != y.h || r.w != y.w)
            return fail(RAFIKI_ERR_INVALID, ln + "residual shape differs from the conv output");
        }
        op.kind = O_CONV;
        op.H = x.h; op.W = x.w; op.Cs_in = x.Cs; op.Ho = Ho; op.Wo = Wo;
        op.kh = L.kh; op.kw = L.kw; op.stride = L.stride; op.pad = L.pad; op.c_out = L.c_out;
        op.cin_l = L.c_in;
        const int c_in = L.c_in, kh = L.kh, kw = L.kw;
        op.K = kh * kw * x.Cs;
        op.Co_pad = bf ? round_up(L.c_out, kCoPadBf16) : round_up(L.c_out, 32);
        op.Kp = bf ? round_up(op.K, 64) : op.K;
        if (e->dry) break;
        auto packed = pack_weight(bf, L.c_out, c_in, kh, kw, x.Cs, op.Co_pad, op.Kp,
                                  [=](int co, int ci, int u, int v) {
                                    return (((size_t)co * c_in + ci) * kh + u) * kw + v;
                                  }, L.weight);
        int rc = upload_gemm_weights(e, op, packed);
        if (!rc) rc = upload_fold(e, op, L);
        if (rc) return rc;
        break;
      }
      case RAFIKI_OP_MAXPOOL2D: {
        if (x.kind != T_IMG) return fail(RAFIKI_ERR_INVALID, ln + "maxpool needs an image tensor");
        if (L.kh < 1 || L.kh != L.kw || L.stride < 1 || L.pad < 0 || L.pad >= L.kh)
          return fail(RAFIKI_ERR_INVALID, ln + "maxpool geometry invalid (square window, pad < k)");
        const int Ho = (x.h + 2 * L.pad - L.kh) / L.stride + 1, Wo = (x.w + 2 * L.pad - L.kw) / L.stride + 1;
        if (x.h + 2 * L.pad < L.kh || x.w + 2 * L.pad < L.kw || Ho < 1 || Wo < 1)
          return fail(RAFIKI_ERR_INVALID, ln + "maxpool output would be empty");
        y = x; y.h = Ho; y.w = Wo; y.off = 0; y.last_use = -1;
        op.kind = O_MAXPOOL; op.H = x.h; op.W = x.w; op.Cs_in = x.Cs; op.Ho = Ho; op.Wo = Wo; op.cin_l = x.c;
        op.k = L.kh; op.stride = L.stride; op.pad = L.pad;
        break;
      }
      case RAFIKI_OP_GLOBAL_AVGPOOL: {
        if (x.kind != T_IMG) return fail(RAFIKI_ERR_INVALID, ln + "global average pool needs an image tensor");
        y.kind = T_VEC; y.c = x.c; y.h = 1; y.w = 1; y.Cs = x.Cs;
        op.kind = O_GAP; op.H = x.h; op.W = x.w; op.Cs_in = x.Cs; op.cin_l = x.c;
        break;
      }
      case RAFIKI_OP_FC: {
        if (x.kind != T_IMG && x.kind != T_VEC) return fail(RAFIKI_ERR_INVALID, ln + "FC needs an image or vector");
        if ((long long)x.c * x.h * x.w != L.c_in || L.c_out < 1 || !L.weight)
          return fail(RAFIKI_ERR_INVALID, ln + "FC c_in must equal the flattened input size");
        if (has_bn) return fail(RAFIKI_ERR_UNSUPPORTED, ln + "batch-norm after FC is not supported");
        y.kind = T_VEC; y.c = L.c_out; y.h = 1; y.w = 1; y.Cs = round_up(L.c_out, 8);
        op.kind = O_CONV;
        op.H = 1; op.W = 1; op.Cs_in = x.h * x.w * x.Cs; op.Ho = 1; op.Wo = 1;
        op.kh = op.kw = op.stride = 1; op.pad = 0; op.c_out = L.c_out;
        op.cin_l = L.c_in;
        op.K = op.Cs_in;
        op.Co_pad = bf ? round_up(L.c_out, kCoPadBf16) : round_up(L.c_out, 32);
        op.Kp = bf ? round_up(op.K, 64) : op.K;
        if (e->dry) break;
        const int xc = x.c, xh = x.h, xw = x.w, xCs = x.Cs, cin = L.c_in;
        // K index (yy, xx, c) over storage channels <- canonical column c*h*w + yy*w + xx
        std::vector<float> packed((size_t)op.Co_pad * op.Kp, 0.f);
        for (int co = 0; co < L.c_out; ++co)
          for (int yy = 0; yy < xh; ++yy)
            for (int xx = 0; xx < xw; ++xx)
              for (int c = 0; c < xc; ++c)
                packed[(size_t)co * op.Kp + (size_t)(yy * xw + xx) * xCs + c] =
                    L.weight[(size_t)co * cin + (size_t)c * xh * xw + yy * xw + xx];
        int rc = upload_gemm_weights(e, op, packed);
        if (!rc) rc = upload_fold(e, op, L);
        if (rc) return rc;
        break;
      }
      case RAFIKI_OP_EMBEDDING: {
        if (L.input != -1 || x.kind != T_TOK) return fail(RAFIKI_ERR_INVALID, ln + "embedding must read the token input");
        if (L.c_in != e->vocab || L.c_out < 1 || !L.weight)
          return fail(RAFIKI_ERR_INVALID, ln + "embedding table must be [vocab, dim]");
        y.kind = T_SEQ; y.c = L.c_out; y.h = 1; y.w = x.w; y.Cs = storage_channels(L.c_out, bf);
        op.kind = O_EMBED; op.Cs_in = y.Cs; op.W = x.w; op.cin_l = L.c_out;
        if (e->dry) break;
        std::vector<float> packed((size_t)L.c_in * y.Cs, 0.f);
        for (int r = 0; r < L.c_in; ++r)
          for (int c = 0; c < L.c_out; ++c) packed[(size_t)r * y.Cs + c] = L.weight[(size_t)r * L.c_out + c];
        int rc = upload_weights(e, op, packed);
        if (rc) return rc;
        break;
      }
      case RAFIKI_OP_CONV1D_MAXTIME: {
        if (x.kind != T_SEQ || L.c_in != x.c || L.c_out < 1 || L.kw < 1 || L.kw > x.w || !L.weight)
          return fail(RAFIKI_ERR_INVALID, ln + "conv1d needs a sequence input with c_in channels and kw <= length");
        y.kind = T_VEC; y.c = L.c_out; y.h = 1; y.w = 1; y.Cs = round_up(L.c_out, 8);
        op.kind = O_CONV1D;
        op.H = 1; op.W = x.w; op.Cs_in = x.Cs; op.Ho = 1; op.Wo = x.w - L.kw + 1;
        op.kh = 1; op.kw = L.kw; op.stride = 1; op.pad = 0; op.c_out = L.c_out;
        op.cin_l = L.c_in;
        op.K = L.kw * x.Cs;
        op.Co_pad = bf ? round_up(L.c_out, kCoPadBf16) : round_up(L.c_out, 32);
        op.Kp = bf ? round_up(op.K, 64) : op.K;
        if (e->dry || in_group[i]) break;   // a fused branch: packed with its group below
        const int cin = L.c_in, kw = L.kw;
        auto packed = pack_weight(bf, L.c_out, cin, 1, kw, x.Cs, op.Co_pad, op.Kp,
                                  [=](int co, int ci, int, int v) { return ((size_t)co * cin + ci) * kw + v; },
                                  L.weight);
        int rc = upload_gemm_weights(e, op, packed);
        if (!rc) rc = upload_fold(e, op, L);
        if (rc) return rc;
        break;
      }
      case RAFIKI_OP_CONCAT: {
        if (L.input2 < 0) return fail(RAFIKI_ERR_INVALID, ln + "concat needs input2");
        const Tensor& b = M.tensors[L.input2];
        if (x.kind != T_VEC || b.kind != T_VEC) return fail(RAFIKI_ERR_INVALID, ln + "concat joins vectors");
        if (L.c_out != x.c + b.c) return fail(RAFIKI_ERR_INVALID, ln + "concat c_out must be the sum of inputs");
        y.kind = T_VEC; y.c = L.c_out; y.h = 1; y.w = 1; y.Cs = round_up(L.c_out, 8);
        op.kind = O_CONCAT; op.ca = x.c; op.cb = b.c;
        break;
      }
      default:
        return fail(RAFIKI_ERR_INVALID, ln + "unknown op " + std::to_string(L.op));
    }
    if (L.op != RAFIKI_OP_CONV2D && L.op != RAFIKI_OP_CONCAT && L.input2 != -1)
      return fail(RAFIKI_ERR_INVALID, ln + "input2 is only meaningful for conv2d and concat");
    if (L.op != RAFIKI_OP_CONV2D && L.op != RAFIKI_OP_FC && L.op != RAFIKI_OP_CONV1D_MAXTIME && op.relu)
      return fail(RAFIKI_ERR_INVALID, ln + "relu is only meaningful for conv2d, FC and conv1d");
    if (L.op != RAFIKI_OP_CONV2D && L.op != RAFIKI_OP_CONV1D_MAXTIME && has_bn && L.op != RAFIKI_OP_FC)
      return fail(RAFIKI_ERR_INVALID, ln + "batch-norm is only meaningful for conv layers");
    M.ops.push_back(op);
  }
  const rafiki_layer& last = md.layers[md.n_layers - 1];
  if (last.op != RAFIKI_OP_FC || last.c_out != md.n_classes)
    return fail(RAFIKI_ERR_INVALID, "model " + std::to_string(mi) + ": the last layer must be an FC with n_classes outputs");
  M.tensors.back().is_logits = true;
  if (!groups.empty()) {
    int rc = fuse_branches(e, md, M, groups);
    if (rc) return rc;
    // A fused GEMM that alone reads an embedding gathers the embedding rows through
    // the token ids itself: the embedded sequence is never stored.
    std::vector<int> readers(M.tensors.size(), 0), writer(M.tensors.size(), -1);
    for (size_t i = 0; i < M.ops.size(); ++i) {
      for (int src : {M.ops[i].in, M.ops[i].in2})
        if (src >= 0) ++readers[src];
      writer[M.ops[i].out] = (int)i;
    }
    std::vector<char> drop(M.ops.size(), 0);
    for (Op& op : M.ops) {
      if (op.nseg == 0 || op.tap_stride == 0 || op.kw > kMaxGatherTaps || op.in < 0 || readers[op.in] != 1) continue;
      const int wi = writer[op.in];
      if (wi < 0 || M.ops[wi].kind != O_EMBED) continue;
      if (e->vocab >= 0xFFFF || (long long)e->vocab * op.Cs_in * (long long)e->esz() >= (1LL << 31)) continue;
      op.table = M.ops[wi].d_w;
      op.in = -1;
      drop[wi] = 1;
    }
    std::vector<Op> kept;
    for (size_t i = 0; i < M.ops.size(); ++i)
      if (!drop[i]) kept.push_back(M.ops[i]);
    M.ops.swap(kept);
  }

  // A 2x2 stride-2 max-pool whose input is a bf16 conv output read by nothing else is
  // fused into that conv: its epilogue writes the pooled tensor, and the full-size conv
  // output is never stored.  ReLU and bf16 rounding are monotone, so the pooled values
  // are bitwise those of the separate pool.
  if (bf) {
    std::vector<int> readers(M.tensors.size(), 0);
    for (const Op& op : M.ops)
      for (int src : {op.in, op.in2})
        if (src >= 0) ++readers[src];
    std::vector<Op> ops;
    std::vector<int> writer(M.tensors.size(), -1);   // index in `ops` of the op writing each tensor
    for (const Op& op : M.ops) {
      if (op.kind == O_MAXPOOL && op.k == 2 && op.stride == 2 && op.pad == 0 && op.in >= 0 &&
          readers[op.in] == 1 && writer[op.in] >= 0) {
        Op& c = ops[writer[op.in]];
        if (c.kind == O_CONV && c.in2 < 0 && !c.pool2 && c.Ho % 2 == 0 && c.Wo % 2 == 0) {
          c.pool2 = 1;
          c.out = op.out;
          writer[op.out] = writer[op.in];
          continue;
        }
      }
      writer[op.out] = (int)ops.size();
      ops.push_back(op);
    }
    M.ops.swap(ops);
  }

  // Liveness-planned arena for max_batch requests (the logits go to the ensemble's slots);
  // a tensor's last use is the index of the last op that reads it.
  for (size_t i = 0; i < M.ops.size(); ++i)
    for (int src : {M.ops[i].in, M.ops[i].in2})
      if (src >= 0) M.tensors[src].last_use = std::max(M.tensors[src].last_use, (int)i);
  FreeList fl;
  const size_t es = e->esz(), nb = (size_t)e->max_batch;
  for (size_t i = 0; i < M.ops.size(); ++i) {
    Op& op = M.ops[i];
    Tensor& y = M.tensors[op.out];
    size_t tmp_bytes = 0;
    if (op.kind == O_CONV1D) {
      tmp_bytes = nb * op.Wo * round_up(op.c_out, 8) * es;
      op.tmp_off = fl.alloc(tmp_bytes);
    }
    if (!y.is_logits) y.off = fl.alloc(nb * y.item_elems() * es);
    if (op.kind == O_CONV1D) fl.release(op.tmp_off, tmp_bytes);
    for (int src : {op.in, op.in2}) {
      if (src >= 0 && M.tensors[src].last_use == (int)i && !M.tensors[src].is_logits)
        fl.release(M.tensors[src].off, nb * M.tensors[src].item_elems() * es);
    }
  }
  M.arena_bytes = std::max<size_t>(fl.top, 256);
  return dev_alloc(e, (void**)&M.d_arena, M.arena_bytes);
}

// Largest split-K partial buffer any GEMM-like op of model M needs for n in [1, max_batch].
size_t partial_need(const rafiki_ensemble_s* e, const Model& M) {
  if (e->precision != RAFIKI_BF16) return 0;
  size_t need = 0;
  for (const Op& op : M.ops) {
    if (op.kind != O_CONV && op.kind != O_CONV1D) continue;
    for (int n = 1; n <= e->max_batch; ++n) {
      const int Mrows = n * op.Ho * op.Wo;
      const int s = choose_splits(Mrows, op.c_out, op.Kp / 64);
      if (s > 1) need = std::max(need, (size_t)s * Mrows * op.Co_pad * 4);
    }
  }
  return need;
}

// The whole-network program of model M (bf16 image models only), or false if a layer
// does not fit the kernel: convolutions 1x1 (pad 0) or 3x3 (pad 1) of stride 1 or 2
// over 8..64 storage channels (a power of two) to at most 64 output channels, with
// Wo a power of two, Ho * Wo a multiple of 32 and no split K at any batch size, then a
// global average pool and the final FC over at most 64 inputs and 32 * kFusedWaves
// classes; the layers' folded scale / shift (copied from the layer kernels' device
// arrays, so bitwise the same) within kFusedTableBytes.  Tensors get
// LDS offsets by liveness; a convolution whose residual is read for the last time
// writes its output over it (each output element replaces the residual element that
// the same lane has just read).  The plan needs at most kFusedLdsBytes.
// LDS arena of one workgroup: live intervals, placed lowest-first (or highest-first)
// in the first gap that fits; sizes rounded to 256 bytes.
struct LdsArena {
  std::vector<std::pair<size_t, size_t>> live;   // (offset, size), sorted by offset
  size_t cap, peak = 0;
  explicit LdsArena(size_t c) : cap(c) {}
  long long place(size_t n, bool high) {
    n = round_up_sz(std::max<size_t>(n, 1), 256);
    long long at = -1;
    if (!high) {
      size_t o = 0;
      for (const auto& iv : live) {
        if (o + n <= iv.first) break;
        o = std::max(o, iv.first + iv.second);
      }
      if (o + n <= cap) at = (long long)o;
    } else {
      long long o = (long long)cap - (long long)n;
      for (auto it = live.rbegin(); it != live.rend(); ++it) {
        if (o >= (long long)(it->first + it->second)) break;
        o = std::min(o, (long long)it->first - (long long)n);
      }
      if (o >= 0) at = o;
    }
    if (at < 0) return -1;
    live.push_back({(size_t)at, n});
    std::sort(live.begin(), live.end());
    peak = std::max(peak, (size_t)at + n);
    return at;
  }
  void release(long long off) {
    for (size_t i = 0; i < live.size(); ++i)
      if ((long long)live[i].first == off) {
        live.erase(live.begin() + i);
        return;
      }
  }
};

// The whole-network program of model M (bf16 image models only), or false if a layer
// does not fit the kernel: convolutions 1x1 (pad 0) or 3x3 (pad 1) of stride 1 or 2
// over 8..64 storage channels (a power of two) to at most 64 output channels, with
// Wo a power of two, Ho * Wo a multiple of 32 and no split K at any batch size, then a
// global average pool and the final FC over at most 64 inputs and 32 * kFusedWaves
// classes; the layers' folded scale / shift (copied from the layer kernels' device
// arrays, so bitwise the same) within kFusedTableBytes.  Tensors get
// LDS offsets by liveness in an arena of kFusedLdsBytes, the model input at its top,
// every other tensor as low as it fits; a convolution whose residual is read for the
// last time writes its output over it (each output element replaces the residual
// element that the same lane has just read).
bool plan_fused(rafiki_ensemble_s* e, Model& M) {
  M.fprog.clear();
  if (e->precision != RAFIKI_BF16 || e->input_kind != RAFIKI_INPUT_IMAGE_NCHW_F32 || !e->fused_net) return false;
  auto cs_ok = [](int cs) { return cs == 8 || cs == 16 || cs == 32 || cs == 64; };
  if (!cs_ok(e->in_Cs) || M.ops.empty()) return false;
  Tensor in_t;
  in_t.kind = T_IMG; in_t.c = e->C; in_t.h = e->H; in_t.w = e->W; in_t.Cs = e->in_Cs;
  auto tens = [&](int id) -> const Tensor& { return id < 0 ? in_t : M.tensors[id]; };
  auto nbytes = [](const Tensor& t) { return (size_t)t.h * t.w * t.Cs * 2; };
  int in_last = -1;
  for (size_t i = 0; i < M.ops.size(); ++i)
    if (M.ops[i].in == -1) in_last = (int)i;
  std::vector<int> writer(M.tensors.size(), -1);
  for (size_t i = 0; i < M.ops.size(); ++i) writer[M.ops[i].out] = (int)i;
  LdsArena ar(kFusedLdsBytes);
  std::vector<long long> off(M.tensors.size(), -1);
  const long long in_off = ar.place(nbytes(in_t), true);
  if (in_off < 0) return false;
  auto loff = [&](int id) { return id < 0 ? in_off : off[id]; };
  std::vector<FusedLayer> prog;
  FusedLayer I{};
  I.op = F_INPUT;
  I.out_off = (int)in_off;
  I.Cso = e->in_Cs;
  I.Ho = e->H; I.Wo = e->W;
  I.ss_off = kFusedLdsBytes + 128;
  prog.push_back(I);
  std::vector<float> table;   // per layer: scale [c4], shift [c4]
  // The weights in fragment order: for channel block cb and K group g, the 64 lanes'
  // 16-byte A fragments (lane fk * 32 + r: row cb * 32 + r, terms 16 g + 8 fk ..
  // + 7) are one contiguous kilobyte, so a wave's fragment load reads whole lines.
  auto frag_weights = [&](FusedLayer& L, const Op& op) -> bool {
    if (e->dry) return true;
    const int NG = (L.K + 15) / 16, rows = L.n_cb * 32;
    std::vector<uint16_t> src((size_t)rows * op.Kp), dst((size_t)L.n_cb * NG * 64 * 8);
    if (hipMemcpy(src.data(), op.d_w, src.size() * 2, hipMemcpyDeviceToHost) != hipSuccess) return false;
    for (int cb = 0; cb < L.n_cb; ++cb)
      for (int g = 0; g < NG; ++g)
        for (int lane = 0; lane < 64; ++lane)
          for (int i = 0; i < 8; ++i)
            dst[(((size_t)cb * NG + g) * 64 + lane) * 8 + i] =
                src[(size_t)(cb * 32 + (lane & 31)) * op.Kp + 16 * g + 8 * (lane >> 5) + i];
    void* d = nullptr;
    if (upload(e, &d, dst.data(), dst.size() * 2)) return false;
    L.w = (const bf16_t*)d;
    return true;
  };
  auto add_table = [&](FusedLayer& L, const Op& op) -> bool {
    const int c4 = (L.c_write + 3) & ~3;
    L.ss_off = I.ss_off + (int)table.size() * 4;
    const size_t at = table.size();
    table.resize(at + 2 * (size_t)c4, 0.f);
    if (e->dry) return true;
    return hipMemcpy(&table[at], op.d_scale, (size_t)L.c_write * 4, hipMemcpyDeviceToHost) == hipSuccess &&
           hipMemcpy(&table[at + c4], op.d_shift, (size_t)L.c_write * 4, hipMemcpyDeviceToHost) == hipSuccess;
  };
  for (size_t i = 0; i < M.ops.size(); ++i) {
    const Op& op = M.ops[i];
    const Tensor& x = tens(op.in);
    const Tensor& y = M.tensors[op.out];
    FusedLayer L{};
    bool aliased = false;
    if (op.kind == O_CONV && !y.is_logits) {
      if (x.kind != T_IMG || op.pool2 || op.kh != op.kw || (op.kh != 1 && op.kh != 3) || op.pad != op.kh / 2 ||
          (op.stride != 1 && op.stride != 2) || !cs_ok(op.Cs_in) || !cs_ok(y.Cs) || op.c_out > 64 ||
          (op.Wo & (op.Wo - 1)) != 0 || (op.Ho * op.Wo) % 32 != 0 || op.Kp / 64 >= 12 ||
          (op.in2 >= 0 && op.in2 == op.in))
        return false;
      L.op = F_CONV;
      L.res_off = -1;
      if (op.in2 >= 0) {
        const Tensor& r = M.tensors[op.in2];
        L.res_off = (int)off[op.in2];
        if (r.last_use == (int)i && nbytes(r) == nbytes(y)) {
          off[op.out] = off[op.in2];
          aliased = true;
        }
      }
      if (!aliased) off[op.out] = ar.place(nbytes(y), false);
      if (off[op.out] < 0) return false;
      L.in_off = (int)loff(op.in);
      L.out_off = (int)off[op.out];
      L.H = op.H; L.W = op.W; L.Cs = op.Cs_in; L.Ho = op.Ho; L.Wo = op.Wo; L.Cso = y.Cs; L.c_write = y.Cs;
      L.kh = op.kh; L.kw = op.kw; L.stride = op.stride; L.pad = op.pad; L.relu = op.relu;
      L.K = op.K; L.Kp = op.Kp;
      L.lwo = 31 - __builtin_clz((unsigned)op.Wo);
      L.n_cb = (y.Cs + 31) / 32;
      L.n_pb = op.Ho * op.Wo / 32;
      // pixel blocks per wave task: enough tasks for every wave, the A fragments reused
      // over up to 4 blocks; a divisor of n_pb
      const int want = std::max(1, std::min(4, L.n_pb * L.n_cb / kFusedWaves));
      L.ch = 1;
      for (int c = 4; c >= 1; c /= 2)
        if (c <= want && L.n_pb % c == 0) { L.ch = c; break; }
    } else if (op.kind == O_GAP) {
      if (x.kind != T_IMG || !cs_ok(op.Cs_in)) return false;
      L.op = F_GAP;
      off[op.out] = ar.place((size_t)op.Cs_in * 2, false);
      if (off[op.out] < 0) return false;
      L.in_off = (int)loff(op.in);
      L.out_off = (int)off[op.out];
      L.H = op.H; L.W = op.W; L.Cs = op.Cs_in;
      // strided partial sums [P][Cs] (fp32) for the block summation order
      const int G = op.Cs_in / 8, P = 256 / std::min(G, 64);
      const long long tmp = ar.place((size_t)P * op.Cs_in * 4, false);
      if (tmp < 0) return false;
      L.tmp_off = (int)tmp;
      ar.release(tmp);
    } else if (op.kind == O_CONV && y.is_logits) {
      if (i + 1 != M.ops.size() || op.in < 0 || writer[op.in] < 0 || M.ops[writer[op.in]].kind != O_GAP ||
          op.Cs_in > 64 || op.K != op.Cs_in || op.c_out > 32 * kFusedWaves || op.Kp / 64 >= 12)
        return false;
      L.op = F_FC;
      L.in_off = (int)off[op.in];
      L.Cs = op.Cs_in; L.K = op.K; L.Kp = op.Kp;
      L.Cso = y.c; L.c_write = y.c; L.relu = op.relu;
      L.n_cb = (op.c_out + 31) / 32;
    } else {
      return false;
    }
    if (L.op != F_GAP && !add_table(L, op)) return false;
    if (L.op != F_GAP && !frag_weights(L, op)) return false;
    if (op.in == -1 && in_last == (int)i) ar.release(in_off);
    for (int src : {op.in, op.in2})
      if (src >= 0 && M.tensors[src].last_use == (int)i && !(aliased && src == op.in2)) ar.release(off[src]);
    prog.push_back(L);
  }
  const size_t tbytes = round_up_sz(table.size() * 4, 16);
  if (ar.peak > (size_t)kFusedLdsBytes || prog.size() + 1 > (size_t)kFusedMaxLayers || tbytes > (size_t)kFusedTableBytes)
    return false;
  table.resize(tbytes / 4, 0.f);
  void* d_table = nullptr;
  if (upload(e, &d_table, table.data(), tbytes)) {
    (void)hipGetLastError();
    return false;
  }
  prog[0].scale = (const float*)d_table;
  prog[0].c_write = (int)tbytes;
  prog.push_back(FusedLayer{});   // F_END
  M.fprog.swap(prog);
  return true;
}

// Algorithmic FLOPs and bytes of model M's forward pass over n requests (the sums of
// its launches' counts; weights read once).
void model_alg(const rafiki_ensemble_s* e, const Model& M, int n, double* flops, double* bytes) {
  const double es = (double)e->esz();
  double f = 0.0, wb = 0.0;
  for (const Op& op : M.ops) {
    if (op.kind != O_CONV) continue;
    const double kalg = (double)op.kh * op.kw * op.cin_l;
    f += 2.0 * n * op.Ho * op.Wo * (double)op.c_out * kalg;
    wb += (double)op.c_out * kalg * es;
  }
  *flops = f;
  *bytes = wb + (double)n * e->H * e->W * e->C * es + (double)n * e->n_classes * 4.0;
}

unsigned magic_div(int d) { return d == 1 ? 0u : (unsigned)((((unsigned long long)1 << 32) + d - 1) / d); }

// Tensor `id` of model M; id -1 is the model input `in` (staged images or the token batch).
const void* tptr(const rafiki_ensemble_s* e, const Model& M, int id, const void* in) {
  (void)e;
  if (id < 0) return in;
  return M.d_arena + M.tensors[id].off;
}

#define HIPCHK(expr)                                                                              \
  do {                                                                                            \
    hipError_t st_ = (expr);                                                                      \
    if (st_ != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(st_)); \
  } while (0)

// Launch `expr` (one kernel launch) on stream s; when tracing, the launch itself records
// a pair of events at the kernel's start and end, and the launch's algorithmic FLOPs
// and bytes are kept with them.
// Tile tuning inside forward passes: while a probe is installed on this thread, every
// conv_mfma launch records a pair of dispatch events (its layer and tile with them).
struct TuneProbe {
  struct Rec { int layer, cfg; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  hipEvent_t next() {
    if (used == pool.size()) {
      hipEvent_t ev = nullptr;
      if (hipEventCreate(&ev) != hipSuccess) return nullptr;
      pool.push_back(ev);
    }
    return pool[used++];
  }
  ~TuneProbe() {
    for (hipEvent_t ev : pool) (void)hipEventDestroy(ev);
  }
};
TuneProbe*& tune_probe() {
  thread_local TuneProbe* p = nullptr;
  return p;
}

// Tile configuration and split count of the GEMM launch being traced (-1 / 0 otherwise).
struct TraceTile { int cfg = -1, splits = 0; };
TraceTile& trace_tile() {
  thread_local TraceTile t;
  return t;
}

// Tile policy of the forward pass being enqueued (set by forward()): 0 the tiles fastest
// alone, 1 the lean tiles, 2 the lean tiles and GEMM tiles for model lean_gemm_model().
int& lean_tiles() {
  thread_local int level = 0;
  return level;
}
int& lean_gemm_model() {
  thread_local int m = -1;
  return m;
}

// A tile of the lean set: 8 waves, at least 128 x 128, K tiles of 64 (one barrier per 64
// of K; the 32-wide tiles of the same footprint gained a third as much alongside other
// models) and a ring of at most 64 KB.
bool lean_cfg(int cfg) {
  if (cfg < 0 || cfg >= kNumMfmaConfigs) return false;
  const MfmaConfig& c = kMfmaConfigs[cfg];
  return c.waves == 8 && c.bm * c.bn >= 128 * 128 && c.bk == 64 &&
         (long long)c.stages * (c.bm + c.bn) * c.bk * 2 <= 64 * 1024;
}

#define TRACED(e, s, kind, model, layer, flops, bytes, expr)                                  \
  do {                                                                                        \
    hipEvent_t ta_ = nullptr, tb_ = nullptr, pa_ = nullptr, pb_ = nullptr;                    \
    if ((e)->trace.on) {                                                                      \
      ta_ = (e)->trace.next();                                                                \
      tb_ = (e)->trace.next();                                                                \
      if (ta_ && tb_) launch_events() = {ta_, tb_};                                           \
    } else if ((kind) == RAFIKI_K_CONV_MFMA && tune_probe()) {                                \
      pa_ = tune_probe()->next();                                                             \
      pb_ = tune_probe()->next();                                                             \
      if (pa_ && pb_) launch_events() = {pa_, pb_};                                           \
    }                                                                                         \
    const hipError_t lst_ = (expr);                                                           \
    launch_events() = {};                                                                     \
    HIPCHK(lst_);                                                                             \
    if (pa_ && pb_) tune_probe()->recs.push_back({(layer), trace_tile().cfg, pa_, pb_});      \
    if (ta_ && tb_)                                                                           \
      (e)->trace.recs.push_back({kind, model, layer, (double)(flops), (double)(bytes), ta_, tb_,     \
                                 trace_tile().cfg, trace_tile().splits});                           \
  } while (0)

// Per-call scratch placed outside the handle (rafiki_ensemble_infer_noalloc): for each
// model, the split-K partial sums of its GEMMs and the keys of its epilogue maxima
// (n rows of ldslot keys per fused op, in op order).  Null when a call uses the
// handle's own buffers.
struct CallScratch {
  float* partial[32] = {};
  size_t partial_bytes[32] = {};
  unsigned* slot[32] = {};
};

// Size limits of the kernels at max_batch, checked by create's validation pass so
// that no infer meets one partway through a forward pass.  The bf16 GEMM addresses its
// input and weights through 32-bit buffer offsets (each below 2 GiB), and every kernel
// numbers the GEMM rows n * Ho * Wo with int.  (A GEMM that gathers embedding rows reads
// only the table, but is checked against the embedded sequence it replaces, which the
// validation pass cannot tell apart.)
int check_limits(const rafiki_ensemble_s* e, int mi, const Model& M) {
  const long long nb = e->max_batch, es = (long long)e->esz();
  for (size_t i = 0; i < M.ops.size(); ++i) {
    const Op& op = M.ops[i];
    if (op.kind != O_CONV && op.kind != O_CONV1D) continue;
    const std::string ln = lname(mi, op.out);
    if (nb * op.Ho * op.Wo >= (1LL << 31))
      return fail(RAFIKI_ERR_UNSUPPORTED, ln + "max_batch * output positions exceeds 2^31 rows; use a smaller max_batch");
    if (e->precision != RAFIKI_BF16) continue;
    if (nb * op.H * op.W * op.Cs_in * es >= (1LL << 31))
      return fail(RAFIKI_ERR_UNSUPPORTED, ln + "the layer's input at max_batch exceeds 2 GiB; use a smaller max_batch");
    if ((long long)op.Co_pad * op.Kp * es >= (1LL << 31))
      return fail(RAFIKI_ERR_UNSUPPORTED, ln + "the layer's weights exceed 2 GiB");
  }
  return RAFIKI_OK;
}

int run_gemm(const rafiki_ensemble_s* e, const Op& op, ConvArgs a, hipStream_t s, int mi, int li, int cfg,
             const CallScratch* ws = nullptr, const int* mis = nullptr) {
  const int nm = a.n_members > 1 ? a.n_members : 1;   // grouped launch: members mis[0 .. nm)
  const double es = (double)e->esz();
  const double kalg = (double)op.kh * op.kw * op.cin_l;
  double flops = 2.0 * a.M * op.c_out * kalg;
  double w_elems = (double)op.c_out * kalg;
  if (op.nseg > 0) {   // fused branches: each branch's own positions and taps
    flops = 0.0;
    w_elems = 0.0;
    for (int i = 0; i < op.nseg; ++i) {
      const double ci = (double)(op.seg_end[i] - (i ? op.seg_end[i - 1] : 0)) * op.seg_kw[i] * op.cin_l;
      flops += 2.0 * a.N * (op.W - op.seg_kw[i] + 1) * ci;
      w_elems += ci;
    }
  }
  const double in_elems = (double)a.N * a.H * a.W * op.cin_l;   // FC: H = W = 1, cin_l = flattened size
  const double out_rows = a.pool2 ? a.M / 4.0 : (double)a.M;
  double bytes = in_elems * es + w_elems * es +
                 (a.maxslot ? 0.0 : out_rows * op.c_out * (a.out_f32 ? 4.0 : es) * (a.res ? 2.0 : 1.0));
  flops *= nm;
  bytes *= nm;
  if (e->precision != RAFIKI_BF16) {
    TRACED(e, s, RAFIKI_K_CONV_F32, mi, li, flops, bytes, launch_conv_f32(a, s));
    return RAFIKI_OK;
  }
  if ((long long)a.N * a.H * a.W * a.Cs * 2 >= (1LL << 31) || (long long)a.Co_pad * a.Kp * 2 >= (1LL << 31))
    return fail(RAFIKI_ERR_UNSUPPORTED, "a layer's input or weights exceed 2 GiB; use a smaller max_batch");
  const int ktiles = a.Kp / 64;
  int splits = choose_splits(a.M, op.c_out, ktiles);
  a.kt_per_split = (ktiles + splits - 1) / splits;
  if (a.tap_stride > 0 && splits > 1) {
    // fused branches: a split takes whole channel blocks, each with the taps of the
    // tile, so that every row's products fall into the same splits whatever the tile
    const int cb = a.Cs / 64, sp = std::min(splits, cb);
    a.kt_per_split = (cb + sp - 1) / sp;
    splits = (cb + a.kt_per_split - 1) / a.kt_per_split;
  }
  if (cfg == kCfgDirect && (splits > 1 || !conv_direct_fits(a))) cfg = -1;   // e.g. a grouped launch
  if (cfg < 0) cfg = splits > 1 ? split_cfg(op.c_out) : default_cfg(op.c_out);
  struct TileScope {
    TileScope(int c, int sp) { trace_tile() = {c, sp}; }
    ~TileScope() { trace_tile() = {}; }
  } tile_scope(cfg, splits);
  if (splits > 1) {
    for (int k = 0; k < nm; ++k) {
      const int m = nm > 1 ? mis[k] : mi;
      const Model& Mo = e->models[m];
      const size_t cap = ws ? ws->partial_bytes[m] : Mo.partial_bytes;
      if ((size_t)splits * a.M * a.Co_pad * 4 > cap)
        return fail(RAFIKI_ERR_INVALID, "internal: split-K workspace too small");
      float* part = ws ? ws->partial[m] : Mo.d_partial;
      if (nm > 1) a.members[k].partial = part;
      else a.partial = part;
    }
    TRACED(e, s, RAFIKI_K_CONV_MFMA, mi, li, flops, bytes, launch_conv_mfma(a, cfg, splits, s));
    TRACED(e, s, RAFIKI_K_SPLITK_REDUCE, mi, li, 0.0,
           nm * ((double)splits * a.M * a.c_write * 4.0 + out_rows * a.c_write * (a.out_f32 ? 4.0 : es)),
           launch_splitk_reduce(a, splits, 1, s));
  } else if (cfg == kCfgDirect) {
    TRACED(e, s, RAFIKI_K_CONV_MFMA, mi, li, flops, bytes, launch_conv_direct(a, s));
  } else {
    TRACED(e, s, RAFIKI_K_CONV_MFMA, mi, li, flops, bytes, launch_conv_mfma(a, cfg, 1, s));
  }
  return RAFIKI_OK;
}

// Whether op (of model M) is one the direct conv kernel takes when launched alone: the
// op-level form of conv_direct_fits (conv_direct.hip) for the tuner's candidate
// list: no residual, and 3x3 stride 1 from 64 to 64 or 128 channels, or (64 output
// channels, with ReLU, no fused pool) 3x3 stride 1 or 7x7 stride 2 over the 8 storage
// channels of an image.
bool direct_op_fits(const rafiki_ensemble_s* e, const Model& M, const Op& op) {
  if (e->precision != RAFIKI_BF16 || op.kind != O_CONV || op.nseg > 0 || op.table || op.in2 >= 0) return false;
  const Tensor& y = M.tensors[op.out];
  if ((op.c_out != 64 && !(op.c_out == 128 && op.Cs_in == 64)) || y.is_logits || y.Cs != op.c_out ||
      op.tap_stride != 0 || op.kh != op.kw || (op.pool2 && (op.Ho % 2 != 0 || op.Wo % 2 != 0)))
    return false;
  auto out_ok = [&](int k, int st) {
    const int pad = k / 2;
    return op.pad == pad && op.stride == st && op.Ho == (op.H + 2 * pad - k) / st + 1 &&
           op.Wo == (op.W + 2 * pad - k) / st + 1;
  };
  if (op.kh == 3 && op.Cs_in == 64 && op.K == 576 && op.Kp == 576 && out_ok(3, 1)) return true;
  if (op.kh == 3 && op.Cs_in == 8 && op.K == 72 && op.Kp >= 80 && op.relu && !op.pool2 && out_ok(3, 1)) return true;
  return op.kh == 7 && op.Cs_in == 8 && op.K == 392 && op.Kp >= 400 && op.relu && !op.pool2 && out_ok(7, 2);
}

// Kernel arguments of a GEMM-like op over n requests (output pointer set by the caller).
ConvArgs gemm_args(const rafiki_ensemble_s* e, const Model& M, const Op& op, int n, const void* in) {
  ConvArgs a{};
  a.x = tptr(e, M, op.in, in); a.w = op.d_w; a.scale = op.d_scale; a.shift = op.d_shift;
  a.res = op.in2 >= 0 ? tptr(e, M, op.in2, in) : nullptr;
  a.N = n; a.H = op.H; a.W = op.W; a.Cs = op.Cs_in;
  a.Ho = op.Ho; a.Wo = op.Wo; a.kh = op.kh; a.kw = op.kw; a.stride = op.stride; a.pad = op.pad;
  a.M = n * op.Ho * op.Wo; a.K = op.K; a.Kp = op.Kp; a.Co_pad = op.Co_pad; a.Nc = op.c_out;
  a.relu = op.relu;
  a.pool2 = op.pool2;
  a.x_bytes = (int)((long long)n * op.H * op.W * op.Cs_in * (long long)e->esz());
  a.w_bytes = (int)((long long)op.Co_pad * op.Kp * (long long)e->esz());
  a.Cs8 = op.Cs_in / 8; a.K8 = op.K / 8;
  a.mag_cs8 = magic_div(op.Cs_in / 8); a.mag_kw = magic_div(op.kw);
  a.tap_stride = op.tap_stride;
  for (int b = 0; b < 16; ++b) a.taps_by_block[b] = op.taps_by_block[b];
  if (op.table) {   // token gather: x is the embedding table, rows picked by the ids
    a.x = op.table;
    a.tok = (const int32_t*)in;
    a.x_bytes = (int)((long long)e->vocab * op.Cs_in * (long long)e->esz());
  }
  return a;
}

int run_models(const rafiki_ensemble_s* e, const int* mis, int nm, const void* in, int n, float* const* logits,
               hipStream_t s, size_t op_begin = 0, size_t op_end = SIZE_MAX, const CallScratch* ws = nullptr);
inline int run_model(const rafiki_ensemble_s* e, int mi, const void* in, int n, float* logits, hipStream_t s,
                     size_t op_begin = 0, size_t op_end = SIZE_MAX, const CallScratch* ws = nullptr) {
  return run_models(e, &mi, 1, in, n, &logits, s, op_begin, op_end, ws);
}

// Choose each GEMM op's tile configuration for batch size n (once per n; blocks the
// caller).  The candidates are timed where they will run: inside forward passes of
// the model on stream s, one model at a time.  Pass j gives every GEMM op its j-th
// candidate; each launch records dispatch events; two rounds of passes, and each op
// keeps the candidate with the shortest launch.  Timed this way a layer reads weights
// that are not in cache and an input the previous layer has just written, as in
// serving (timing a candidate by repeating it alone kept the weights in L2 and chose
// shallow pipelines that are slower in the pass).  All candidates sum K in the same
// order, and a split-K launch keeps the split that the shape fixes (only its tile is
// tuned), so the choice never changes a result.
int tune(rafiki_ensemble_s* e, int n, const void* in, hipStream_t s) {
  if (e->tuned.count(n)) return RAFIKI_OK;
  const size_t NM = e->models.size();
  std::vector<std::vector<int>> choice(NM);
  std::vector<std::vector<std::vector<int>>> cand(NM);
  std::vector<double> est(NM, 0.0);
  bool all_fused = e->d_fprog != nullptr;
  for (const Model& M : e->models) all_fused = all_fused && !M.fprog.empty();
  const bool timing = e->autotune && e->precision == RAFIKI_BF16 && !all_fused;
  for (size_t mi = 0; mi < NM; ++mi) {
    const Model& M = e->models[mi];
    choice[mi].assign(M.ops.size(), -1);
    cand[mi].resize(M.ops.size());
    for (size_t oi = 0; oi < M.ops.size(); ++oi) {
      const Op& op = M.ops[oi];
      if (op.kind != O_CONV && op.kind != O_CONV1D) continue;
      const int M_rows = n * op.Ho * op.Wo;
      const int splits = choose_splits(M_rows, op.c_out, op.Kp / 64);
      choice[mi][oi] = splits > 1 ? split_cfg(op.c_out) : default_cfg(op.c_out);
      est[mi] += 2.0 * n * op.Ho * op.Wo * (double)op.c_out * op.K / 1e12;
      if (!timing) continue;
      for (int cfg = 0; cfg < kNumMfmaConfigs; ++cfg)
        if (cfg_fits(cfg, op.c_out) && kMfmaConfigs[cfg].bm <= 2 * round_up(M_rows, 32)) cand[mi][oi].push_back(cfg);
      if (splits == 1 && direct_op_fits(e, M, op)) cand[mi][oi].push_back(kCfgDirect);
    }
  }
  if (!timing) {
    e->tuned_lean[n] = choice;
    e->tuned_lean_gemm[n] = choice;
    e->tuned[n] = std::move(choice);
    e->model_ms[n] = std::move(est);
    return RAFIKI_OK;
  }
  // best[mi][oi][cfg]: shortest launch seen.  A forced tile and the caller's tracing
  // are suspended during the passes.
  std::vector<std::vector<std::vector<float>>> best(NM);
  TuneProbe probe;
  int rc = RAFIKI_OK;
  const int saved_force = e->force_tile;
  const bool saved_trace = e->trace.on;
  e->force_tile = -1;
  e->trace.on = false;
  for (size_t mi = 0; mi < NM && rc == RAFIKI_OK; ++mi) {
    const Model& M = e->models[mi];
    best[mi].assign(M.ops.size(), std::vector<float>(kNumMfmaConfigs + 1, 1e30f));
    std::vector<int> out_to_op(M.tensors.size(), -1);
    size_t J = 0;
    for (size_t oi = 0; oi < M.ops.size(); ++oi) {
      out_to_op[M.ops[oi].out] = (int)oi;
      J = std::max(J, cand[mi][oi].size());
    }
    float* logits = e->d_logits + mi * (size_t)e->max_batch * e->n_classes;
    for (int round = 0; round < 2 && rc == RAFIKI_OK; ++round)
      for (size_t j = 0; j < J && rc == RAFIKI_OK; ++j) {
        std::vector<std::vector<int>> pass = choice;
        for (size_t oi = 0; oi < M.ops.size(); ++oi)
          if (!cand[mi][oi].empty()) pass[mi][oi] = cand[mi][oi][j % cand[mi][oi].size()];
        e->tuned[n] = std::move(pass);
        probe.recs.clear();
        probe.used = 0;
        tune_probe() = &probe;
        rc = run_model(e, (int)mi, in, n, logits, s, 0, SIZE_MAX);
        tune_probe() = nullptr;
        if (rc) break;
        for (const TuneProbe::Rec& r : probe.recs) {
          float ms = 0.f;
          hipError_t st = hipEventSynchronize(r.b);
          if (st == hipSuccess) st = hipEventElapsedTime(&ms, r.a, r.b);
          if (st != hipSuccess) {
            rc = fail(RAFIKI_ERR_HIP, std::string("tile tuning timing: ") + hipGetErrorString(st));
            break;
          }
          const int oi = r.layer >= 0 && r.layer < (int)out_to_op.size() ? out_to_op[r.layer] : -1;
          if (oi >= 0 && r.cfg >= 0 && r.cfg <= kCfgDirect)
            best[mi][oi][r.cfg] = std::min(best[mi][oi][r.cfg], ms);
        }
      }
  }
  e->tuned.erase(n);
  e->force_tile = saved_force;
  e->trace.on = saved_trace;
  if (rc) return rc;
  std::vector<std::vector<int>> lean(NM);
  for (size_t mi = 0; mi < NM; ++mi) {
    est[mi] = 0.0;
    lean[mi] = choice[mi];
    for (size_t oi = 0; oi < cand[mi].size(); ++oi) {
      float t = 1e30f;
      for (int cfg : cand[mi][oi])
        if (best[mi][oi][cfg] < t) { t = best[mi][oi][cfg]; choice[mi][oi] = cfg; }
      if (t < 1e29f) est[mi] += t;
      const Op& op = e->models[mi].ops[oi];
      lean[mi][oi] = choice[mi][oi];
      if (op.Ho * op.Wo > 196 || op.Ho * op.Wo < 2 || choose_splits(n * op.Ho * op.Wo, op.c_out, op.Kp / 64) > 1)
        continue;
      float tl = 1e30f;
      for (int cfg : cand[mi][oi])
        if (lean_cfg(cfg) && best[mi][oi][cfg] < tl) { tl = best[mi][oi][cfg]; lean[mi][oi] = cfg; }
    }
  }
  std::vector<std::vector<int>> lean_gemm = lean;
  for (size_t mi = 0; mi < NM; ++mi)
    for (size_t oi = 0; oi < cand[mi].size(); ++oi) {
      if (lean_gemm[mi][oi] != kCfgDirect) continue;
      const Op& op = e->models[mi].ops[oi];
      float t = 1e30f;
      int pick = default_cfg(op.c_out);
      for (int cfg : cand[mi][oi])
        if (cfg != kCfgDirect && best[mi][oi][cfg] < t) { t = best[mi][oi][cfg]; pick = cfg; }
      lean_gemm[mi][oi] = pick;
    }
  e->tuned_lean_gemm[n] = std::move(lean_gemm);
  e->tuned_lean[n] = std::move(lean);
  e->tuned[n] = std::move(choice);
  e->model_ms[n] = std::move(est);
  return RAFIKI_OK;
}

// Forward pass of model `mi` over n requests whose model input is `in` (staged images
// or token ids); logits [n][n_classes] to `logits`.  Several models with identical
// layer lists (mis[0 .. nm), nm <= kMaxGroup) run as one grouped launch per op, member
// k writing its logits to logits[k]; ops without a grouped kernel (embedding gather,
// concatenation) are launched once per member.
// Only ops [op_begin, op_end) are enqueued, so that the launches of several models
// can be interleaved.
// One op of several members in one launch: member k is op ois[k] of model mis[k]; every
// member's op has the same launch signature (same_launch), so the launch shares shapes,
// tile and K splits and each member's outputs are those of its own launch.  The tile
// is member 0's tuned one (every tile gives the same sums).
int run_op(const rafiki_ensemble_s* e, const int* mis, const int* ois, int nm, const void* in, int n,
           float* const* logits, hipStream_t s, const CallScratch* ws) {
  if (nm < 1 || nm > kMaxGroup) return fail(RAFIKI_ERR_INVALID, "internal: group size");
  const int mi = mis[0];
  const Model& M = e->models[mi];
  const auto& table = lean_tiles() == 2 && mi == lean_gemm_model() ? e->tuned_lean_gemm
                      : lean_tiles() ? e->tuned_lean : e->tuned;
  const auto it = table.find(n);
  const std::vector<int> empty;
  const std::vector<int>& cfgs = it == table.end() ? empty : it->second[mi];
  const int bf = e->precision == RAFIKI_BF16 ? 1 : 0;
  const double es = (double)e->esz();
  const size_t oi = (size_t)ois[0];
  {
    const Op& op = M.ops[oi];
    const int li = op.out;
    // member k's op, tensors and pointers (k = 0 is model mi)
    auto mop = [&](int k) -> const Op& { return e->models[mis[k]].ops[ois[k]]; };
    auto yptr = [&](int k) -> void* {
      const Model& Mk = e->models[mis[k]];
      const Tensor& y = Mk.tensors[Mk.ops[ois[k]].out];
      return y.is_logits ? (void*)logits[k] : (void*)(Mk.d_arena + y.off);
    };
    auto xptr = [&](int k, int id) { return tptr(e, e->models[mis[k]], id, in); };
    // this op's epilogue-max keys of member k (ws: after those of the model's earlier fused ops)
    auto slotptr = [&](int k) -> unsigned* {
      const Model& Mk = e->models[mis[k]];
      if (!ws) return Mk.ops[ois[k]].d_slot;
      unsigned* p = ws->slot[mis[k]];
      for (int j = 0; j < ois[k]; ++j)
        if (Mk.ops[j].d_slot) p += (size_t)n * Mk.ops[j].ldslot;
      return p;
    };
    void* yp = yptr(0);
    const Tensor& y = M.tensors[op.out];
    switch (op.kind) {
      case O_CONV:
      case O_CONV1D: {
        ConvArgs a = gemm_args(e, M, op, n, in);
        int cfg = cfgs.empty() ? -1 : cfgs[oi];
        if (e->force_tile == kCfgDirect) {
          if (direct_op_fits(e, M, op)) cfg = kCfgDirect;
        } else if (e->force_tile >= 0 && cfg_fits(e->force_tile, op.c_out)) {
          cfg = e->force_tile;
        }
        if (nm > 1) {
          a.n_members = nm;
          for (int k = 0; k < nm; ++k) {
            const Op& ok = mop(k);
            GroupMember& g = a.members[k];
            g.x = ok.table ? ok.table : xptr(k, ok.in);
            g.w = ok.d_w;
            g.scale = ok.d_scale;
            g.shift = ok.d_shift;
            g.res = ok.in2 >= 0 ? xptr(k, ok.in2) : nullptr;
          }
        }
        if (op.kind == O_CONV1D) {
          void* tmp = M.d_arena + op.tmp_off;
          a.y = tmp; a.c_write = round_up(op.c_out, 8); a.ldy = a.c_write; a.out_f32 = bf ? 0 : 1;
          const bool in_epilogue = op.d_slot && choose_splits(a.M, op.c_out, a.Kp / 64) == 1;
          GroupIO fin{};   // per member: slots, pre-max rows and the concatenated vector
          fin.n = nm;
          for (int k = 0; k < nm; ++k) {
            const Model& Mk = e->models[mis[k]];
            fin.slot[k] = slotptr(k);
            fin.x[k] = Mk.d_arena + mop(k).tmp_off;
            fin.y[k] = yptr(k);
            if (nm > 1) {
              a.members[k].y = (void*)fin.x[k];
              a.members[k].maxslot = in_epilogue ? fin.slot[k] : nullptr;
            }
          }
          if (in_epilogue) { a.maxslot = fin.slot[0]; a.ldslot = op.ldslot; }
          int rc = run_gemm(e, op, a, s, mi, li, cfg, ws, mis);
          if (rc) return rc;
          if (in_epilogue) {   // the GEMM took the max; write the concatenated vector
            ReduceSegs segs{};
            segs.n = op.nseg; segs.ldy = y.Cs; segs.zero_from = y.c;
            for (int i = 0; i < op.nseg; ++i) {
              segs.dst[i] = i ? op.seg_end[i - 1] : 0;
              segs.cnt[i] = op.seg_end[i] - segs.dst[i];
              segs.src[i] = op.seg_row[i];
              segs.len[i] = op.W - op.seg_kw[i] + 1;
            }
            TRACED(e, s, RAFIKI_K_POOL, mi, li, 0.0,
                   nm * ((double)n * op.ldslot * 4.0 * 2.0 + (double)n * y.Cs * es),
                   launch_maxslot_finish(fin, op.ldslot, n, segs, s));
            break;
          }
          ReduceSegs segs{};
          double vals = (double)op.Wo * op.c_out;   // pre-max values read per request
          if (op.nseg > 0) {
            segs.n = op.nseg;
            segs.ldy = y.Cs;
            segs.zero_from = y.c;
            vals = 0.0;
            for (int i = 0; i < op.nseg; ++i) {
              segs.dst[i] = i ? op.seg_end[i - 1] : 0;
              segs.cnt[i] = op.seg_end[i] - segs.dst[i];
              segs.src[i] = op.seg_row[i];
              segs.len[i] = op.W - op.seg_kw[i] + 1;
              vals += (double)segs.len[i] * segs.cnt[i];
            }
          }
          TRACED(e, s, RAFIKI_K_POOL, mi, li, 0.0, nm * ((double)n * vals * es + (double)n * y.c * es),
                 launch_spatial_reduce(fin, n, op.Wo, a.c_write, 1, bf, s, op.nseg > 0 ? &segs : nullptr));
          break;
        }
        a.y = yp;
        if (nm > 1)
          for (int k = 0; k < nm; ++k) a.members[k].y = yptr(k);
        if (y.is_logits) { a.c_write = y.c; a.ldy = y.c; a.out_f32 = 1; }
        else { a.c_write = y.Cs; a.ldy = y.Cs; a.out_f32 = bf ? 0 : 1; }
        int rc = run_gemm(e, op, a, s, mi, li, cfg, ws, mis);
        if (rc) return rc;
        break;
      }
      case O_MAXPOOL:
      case O_GAP: {
        GroupIO io{};
        io.n = nm;
        for (int k = 0; k < nm; ++k) {
          io.x[k] = xptr(k, mop(k).in);
          io.y[k] = yptr(k);
        }
        if (op.kind == O_MAXPOOL)
          TRACED(e, s, RAFIKI_K_POOL, mi, li, 0.0,
                 nm * ((double)op.H * op.W + (double)op.Ho * op.Wo) * n * op.cin_l * es,
                 launch_maxpool(io, n, op.H, op.W, op.Cs_in, op.Ho, op.Wo, op.k, op.stride, op.pad, bf, s));
        else
          TRACED(e, s, RAFIKI_K_POOL, mi, li, 0.0, nm * ((double)op.H * op.W + 1.0) * n * op.cin_l * es,
                 launch_spatial_reduce(io, n, op.H * op.W, op.Cs_in, 0, bf, s));
        break;
      }
      case O_EMBED:
        for (int k = 0; k < nm; ++k)
          TRACED(e, s, RAFIKI_K_EMBED, mis[k], li, 0.0, (double)n * op.W * (4.0 + 2.0 * op.cin_l * es),
                 launch_embed_gather((const int32_t*)in, mop(k).d_w, yptr(k), n, op.W, op.Cs_in, e->vocab, bf, s));
        break;
      case O_CONCAT:
        for (int k = 0; k < nm; ++k) {
          const Model& Mk = e->models[mis[k]];
          const Tensor& ta = Mk.tensors[op.in];
          const Tensor& tb = Mk.tensors[op.in2];
          TRACED(e, s, RAFIKI_K_CONCAT, mis[k], li, 0.0, 2.0 * n * (op.ca + op.cb) * es,
                 launch_concat(xptr(k, op.in), op.ca, ta.Cs, xptr(k, op.in2), op.cb, tb.Cs, yptr(k), Mk.tensors[op.out].Cs,
                               n, bf, s));
        }
        break;
    }
  }
  return RAFIKI_OK;
}

int run_models(const rafiki_ensemble_s* e, const int* mis, int nm, const void* in, int n, float* const* logits,
               hipStream_t s, size_t op_begin, size_t op_end, const CallScratch* ws) {
  if (nm < 1 || nm > kMaxGroup) return fail(RAFIKI_ERR_INVALID, "internal: group size");
  op_end = std::min(op_end, e->models[mis[0]].ops.size());
  for (size_t oi = op_begin; oi < op_end; ++oi) {
    int ois[kMaxGroup];
    for (int k = 0; k < nm; ++k) ois[k] = (int)oi;
    const int rc = run_op(e, mis, ois, nm, in, n, logits, s, ws);
    if (rc) return rc;
  }
  return RAFIKI_OK;
}

int check_call(const rafiki_ensemble_s* h, const void* batch, int n) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (!batch) return fail(RAFIKI_ERR_INVALID, "null batch pointer");
  if (n < 1 || n > h->max_batch)
    return fail(RAFIKI_ERR_INVALID, "n must be in [1, max_batch = " + std::to_string(h->max_batch) + "]");
  return RAFIKI_OK;
}

// The forward passes' input: the staging buffer for images, the batch itself for tokens.
const void* model_input(const rafiki_ensemble_s* e, const void* batch, void* staged) {
  return e->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32 ? staged : batch;
}

int stage(const rafiki_ensemble_s* e, const void* batch, int n, hipStream_t s, void* dst) {
  if (e->input_kind != RAFIKI_INPUT_IMAGE_NCHW_F32) return RAFIKI_OK;
  TRACED(e, s, RAFIKI_K_STAGE, -1, -1, 0.0, (double)n * e->C * e->H * e->W * (4.0 + (double)e->esz()),
         launch_stage_images((const float*)batch, dst, n, e->C, e->H, e->W, e->in_Cs,
                             e->precision == RAFIKI_BF16, s));
  return RAFIKI_OK;
}

}  // namespace

namespace rafiki {
int set_error(int code, const std::string& msg) { return fail(code, msg); }

// Two models whose layer lists differ only in their parameters: every op and tensor
// has the same kind, wiring, shapes, padding, tiling fields and arena offsets.
bool same_structure(const Model& A, const Model& B) {
  if (A.ops.size() != B.ops.size() || A.tensors.size() != B.tensors.size() || A.arena_bytes != B.arena_bytes)
    return false;
  for (size_t i = 0; i < A.tensors.size(); ++i) {
    const Tensor &a = A.tensors[i], &b = B.tensors[i];
    if (a.kind != b.kind || a.c != b.c || a.h != b.h || a.w != b.w || a.Cs != b.Cs || a.off != b.off ||
        a.is_logits != b.is_logits)
      return false;
  }
  for (size_t i = 0; i < A.ops.size(); ++i) {
    const Op &a = A.ops[i], &b = B.ops[i];
    const int fa[] = {a.kind, a.in, a.in2, a.out, a.H, a.W, a.Cs_in, a.Ho, a.Wo, a.kh, a.kw, a.stride, a.pad, a.relu,
                      a.K, a.Kp, a.Co_pad, a.c_out, a.cin_l, a.k, a.pool2, a.nseg, a.tap_stride, a.ldslot, a.ca, a.cb,
                      a.table != nullptr, a.d_slot != nullptr};
    const int fb[] = {b.kind, b.in, b.in2, b.out, b.H, b.W, b.Cs_in, b.Ho, b.Wo, b.kh, b.kw, b.stride, b.pad, b.relu,
                      b.K, b.Kp, b.Co_pad, b.c_out, b.cin_l, b.k, b.pool2, b.nseg, b.tap_stride, b.ldslot, b.ca, b.cb,
                      b.table != nullptr, b.d_slot != nullptr};
    if (std::memcmp(fa, fb, sizeof(fa)) != 0 || a.tmp_off != b.tmp_off) return false;
    for (int j = 0; j < kMaxReduceSegs; ++j)
      if (a.seg_end[j] != b.seg_end[j] || a.seg_kw[j] != b.seg_kw[j] || a.seg_row[j] != b.seg_row[j]) return false;
    for (int j = 0; j < 16; ++j)
      if (a.taps_by_block[j] != b.taps_by_block[j]) return false;
  }
  return true;
}

// Two ops whose launches can be one launch with a member each: the same kind, shapes,
// K layout, padding, epilogue and output tensor layout (the tensors themselves differ).
bool same_op(const Model& A, const Op& a, const Model& B, const Op& b) {
  const Tensor &ya = A.tensors[a.out], &yb = B.tensors[b.out];
  const int fa[] = {a.kind, a.H, a.W, a.Cs_in, a.Ho, a.Wo, a.kh, a.kw, a.stride, a.pad, a.relu, a.K, a.Kp, a.Co_pad,
                    a.c_out, a.cin_l, a.k, a.pool2, a.nseg, a.tap_stride, a.ldslot, a.ca, a.cb, a.in2 >= 0,
                    a.table != nullptr, a.d_slot != nullptr, ya.kind, ya.c, ya.h, ya.w, ya.Cs, ya.is_logits};
  const int fb[] = {b.kind, b.H, b.W, b.Cs_in, b.Ho, b.Wo, b.kh, b.kw, b.stride, b.pad, b.relu, b.K, b.Kp, b.Co_pad,
                    b.c_out, b.cin_l, b.k, b.pool2, b.nseg, b.tap_stride, b.ldslot, b.ca, b.cb, b.in2 >= 0,
                    b.table != nullptr, b.d_slot != nullptr, yb.kind, yb.c, yb.h, yb.w, yb.Cs, yb.is_logits};
  if (std::memcmp(fa, fb, sizeof(fa)) != 0 || a.nseg != 0 || a.kind == O_EMBED || a.kind == O_CONCAT) return false;
  return true;
}

// The merged op order of two models: a longest common subsequence of their ops under
// same_op (aligned steps), with each model's other ops in between in their own order.
std::vector<std::pair<int, int>> align_ops(const Model& A, const Model& B) {
  const int na = (int)A.ops.size(), nb = (int)B.ops.size();
  std::vector<std::vector<int>> L(na + 1, std::vector<int>(nb + 1, 0));
  for (int i = na - 1; i >= 0; --i)
    for (int j = nb - 1; j >= 0; --j)
      L[i][j] = same_op(A, A.ops[i], B, B.ops[j]) ? L[i + 1][j + 1] + 1 : std::max(L[i + 1][j], L[i][j + 1]);
  std::vector<std::pair<int, int>> steps;
  int i = 0, j = 0;
  while (i < na || j < nb) {
    if (i < na && j < nb && same_op(A, A.ops[i], B, B.ops[j]) && L[i][j] == L[i + 1][j + 1] + 1) {
      steps.push_back({i++, j++});
    } else if (j >= nb || (i < na && L[i + 1][j] >= L[i][j + 1])) {
      steps.push_back({i++, -1});
    } else {
      steps.push_back({-1, j++});
    }
  }
  return steps;
}

// Scratch of rafiki_ensemble_infer_noalloc: a file-scope device array, one copy per
// GPU, held until the process ends.  Host code never uses the array's name as an
// address (on the host it is only a stand-in for the symbol): each device's address
// comes from hipGetSymbolAddress, taken once per device by scratch_on_device().
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxScratchDevices = 64;

// Address of `scratch` on the current device, resolved on the first call for that
// device (with it current) and kept; null with *err set if the device index is out
// of range or the lookup failed (the failure is kept too and reported again).
void* scratch_on_device(int device, std::string* err) {
  static std::mutex mu;
  static void* ptr[kMaxScratchDevices] = {};
  static std::string why[kMaxScratchDevices];
  static bool done[kMaxScratchDevices] = {};
  if (device < 0 || device >= kMaxScratchDevices) {
    *err = "device index " + std::to_string(device) + " beyond the scratch table";
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!done[device]) {
    void* p = nullptr;
    const hipError_t st = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (st != hipSuccess || !p) {
      (void)hipGetLastError();
      why[device] = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(st);
      p = nullptr;
    }
    ptr[device] = p;
    done[device] = true;
  }
  if (!ptr[device]) *err = why[device];
  return ptr[device];
}

__global__ void zero_u32_kernel(unsigned* p, long long count) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) p[i] = 0u;
}
}  // namespace rafiki

extern "C" {

int rafiki_ensemble_create(const rafiki_model_desc* models, int n_models, const rafiki_ensemble_opts* opts,
                           rafiki_ensemble_t* out) {
  if (out) *out = nullptr;
  if (!models || !opts || !out) return fail(RAFIKI_ERR_INVALID, "null argument");
  if (n_models < 1 || n_models > 32) return fail(RAFIKI_ERR_INVALID, "n_models must be in [1, 32]");
  if (opts->precision != RAFIKI_FP32 && opts->precision != RAFIKI_BF16)
    return fail(RAFIKI_ERR_INVALID, "unknown precision");
  if (opts->max_batch < 1) return fail(RAFIKI_ERR_INVALID, "max_batch must be >= 1");
  if (opts->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32) {
    if (opts->c < 1 || opts->h < 1 || opts->w < 1) return fail(RAFIKI_ERR_INVALID, "image shape must be positive");
  } else if (opts->input_kind == RAFIKI_INPUT_TOKENS_I32) {
    if (opts->h < 1 || opts->vocab < 1) return fail(RAFIKI_ERR_INVALID, "sequence length and vocab must be positive");
  } else {
    return fail(RAFIKI_ERR_INVALID, "unknown input kind");
  }
  const int n_classes = models[0].n_classes;
  for (int m = 0; m < n_models; ++m)
    if (models[m].n_classes != n_classes)
      return fail(RAFIKI_ERR_INVALID, "all models must have the same number of classes");
  if (n_classes > 1024) return fail(RAFIKI_ERR_UNSUPPORTED, "at most 1024 classes are supported");

  std::unique_ptr<rafiki_ensemble_s> e(new rafiki_ensemble_s());
  e->n_models = n_models; e->n_classes = n_classes; e->precision = opts->precision;
  e->max_batch = opts->max_batch; e->input_kind = opts->input_kind;
  e->C = opts->c; e->H = opts->h; e->W = opts->w; e->vocab = opts->vocab;
  if (e->input_kind == RAFIKI_INPUT_TOKENS_I32) { e->C = 1; e->W = 1; }
  e->in_Cs = round_up(e->C, 8);
  if (const char* t = std::getenv("RAFIKI_AUTOTUNE")) e->autotune = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_MODEL_STREAMS")) e->concurrent = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_GRAPHS")) e->use_graphs = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_SCHEDULE_TUNING")) e->tune_schedule = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_FUSE_BRANCHES")) e->fuse_branches = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_LEAN_TILES")) e->lean_policy = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_GROUPED")) e->grouped = std::atoi(t) != 0;
  if (const char* t = std::getenv("RAFIKI_FUSED_NET")) e->fused_net = std::atoi(t) != 0;
  // Pass 1: validate every model and infer shapes without touching the device.
  e->dry = true;
  e->models.resize(n_models);
  for (int m = 0; m < n_models; ++m) {
    int rc = build_model(e.get(), m, models[m], e->models[m]);
    if (!rc) rc = check_limits(e.get(), m, e->models[m]);
    if (rc) return rc;
  }
  int ndev = 0;
  hipError_t st = hipGetDeviceCount(&ndev);
  if (st != hipSuccess || ndev < 1) {
    (void)hipGetLastError();
    return fail(RAFIKI_ERR_HIP, std::string("no HIP device: ") + hipGetErrorString(st));
  }
  st = hipGetDevice(&e->device);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(st));
  // Pass 2: pack and upload.
  e->dry = false;
  e->models.clear();
  e->models.resize(n_models);
  for (int m = 0; m < n_models; ++m) {
    int rc = build_model(e.get(), m, models[m], e->models[m]);
    if (rc) return rc;
  }
  e->group_of.resize(n_models);
  for (int m = 0; m < n_models; ++m) {
    e->group_of[m] = m;
    for (int j = 0; j < m; ++j)
      if (same_structure(e->models[j], e->models[m])) {
        e->group_of[m] = j;
        break;
      }
  }
  // Pairable models: bf16, different layer lists, at least half of the shorter one's
  // ops aligned with ops of the other.
  if (e->precision == RAFIKI_BF16)
    for (int a = 0; a < n_models; ++a)
      for (int b = a + 1; b < n_models; ++b) {
        if (e->group_of[a] == e->group_of[b]) continue;
        std::vector<std::pair<int, int>> steps = align_ops(e->models[a], e->models[b]);
        size_t matched = 0;
        for (const auto& st : steps) matched += st.first >= 0 && st.second >= 0;
        if (2 * matched >= std::min(e->models[a].ops.size(), e->models[b].ops.size()))
          e->pairing[{a, b}] = std::move(steps);
      }
  int rc;
  {   // whole-network programs of the models that fit the kernel
    std::vector<FusedLayer> progs((size_t)n_models * kFusedMaxLayers, FusedLayer{});
    bool any = false;
    for (int m = 0; m < n_models; ++m)
      if (plan_fused(e.get(), e->models[m])) {
        std::copy(e->models[m].fprog.begin(), e->models[m].fprog.end(), progs.begin() + (size_t)m * kFusedMaxLayers);
        any = true;
      }
    if (any) {
      rc = upload(e.get(), (void**)&e->d_fprog, progs.data(), progs.size() * sizeof(FusedLayer));
      if (rc) return rc;
    }
  }
  if (e->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32) {
    rc = dev_alloc(e.get(), &e->d_staged, (size_t)e->max_batch * e->H * e->W * e->in_Cs * e->esz());
    if (rc) return rc;
  }
  rc = dev_alloc(e.get(), (void**)&e->d_logits, (size_t)n_models * e->max_batch * n_classes * 4);
  if (rc) return rc;
  for (int mi = 0; mi < n_models; ++mi) {
    Model& M = e->models[mi];
    M.partial_bytes = partial_need(e.get(), M);
    if (M.partial_bytes) {
      rc = dev_alloc(e.get(), (void**)&M.d_partial, M.partial_bytes);
      if (rc) return rc;
    }
    hipError_t st2 = hipStreamCreateWithFlags(&M.stream, hipStreamNonBlocking);
    if (st2 == hipSuccess) st2 = hipEventCreateWithFlags(&M.done, hipEventDisableTiming);
    if (st2 != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("stream/event creation: ") + hipGetErrorString(st2));
  }
  if (e->input_kind == RAFIKI_INPUT_TOKENS_I32) {
    rc = dev_alloc(e.get(), &e->d_tokens, (size_t)e->max_batch * e->H * 4);
    if (rc) return rc;
  }
  // the no-alloc variant's scratch on this device (a failure only disables that call)
  e->scratch = scratch_on_device(e->device, &e->scratch_err);
  {
    hipError_t st2 = hipEventCreateWithFlags(&e->staged_ev, hipEventDisableTiming);
    if (st2 == hipSuccess) st2 = hipStreamCreateWithFlags(&e->capture_stream, hipStreamNonBlocking);
    if (st2 != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("event creation: ") + hipGetErrorString(st2));
  }
  *out = e.release();
  g_err.clear();
  return RAFIKI_OK;
}

}  // extern "C"

// Forward passes of the models ca.sel over n requests whose model input is `in`, logits
// into the workspace, ordered after the work already on s and before what follows it.
// Selected models are independent until the combine: they fork onto their own streams
// and join back (sequential when tracing, so that each traced kernel has the GPU to
// itself).  Forked launches are enqueued interleaved, one op of each model in turn, so
// that every model stream has work from the start even when enqueueing is slower than
// the device.
// The selection runs as grouped launches: two or more models of one group.
static bool grouped_selection(const rafiki_ensemble_s* h, const CombineArgs& ca) {
  if (!h->grouped || ca.S < 2) return false;
  for (int i = 1; i < ca.S; ++i)
    if (h->group_of[ca.sel[i]] != h->group_of[ca.sel[0]]) return false;
  return true;
}

// Model m runs as the whole-network kernel.
static bool fused_model(const rafiki_ensemble_s* h, int m) { return h->d_fprog && !h->models[m].fprog.empty(); }
static bool fused_selection(const rafiki_ensemble_s* h, const CombineArgs& ca) {
  for (int i = 0; i < ca.S; ++i)
    if (!fused_model(h, ca.sel[i])) return false;
  return ca.S > 0;
}

// One launch of the whole-network kernel: the models of `mask` over n staged images,
// model m's logits at logits + m * ld_model.
static int run_fused(const rafiki_ensemble_s* h, uint32_t mask, const void* in, int n, float* logits,
                     long long ld_model, hipStream_t s) {
  FusedNetArgs a{};
  a.progs = h->d_fprog;
  a.logits = logits;
  a.ld_model = ld_model;
  a.mask = mask;
  a.in = (const bf16_t*)in;
  double flops = 0.0, bytes = 0.0;
  for (int m = 0; m < h->n_models; ++m)
    if ((mask >> m) & 1u) {
      double f, b;
      model_alg(h, h->models[m], n, &f, &b);
      flops += f;
      bytes += b;
    }
  TRACED(h, s, RAFIKI_K_FUSED_NET, -1, -1, flops, bytes, launch_fused_net(a, n, __builtin_popcount(mask), s));
  return RAFIKI_OK;
}

// The pairing of the selection's models pa and pb, or null.
static const std::vector<std::pair<int, int>>* selected_pairing(const rafiki_ensemble_s* h, const CombineArgs& ca,
                                                                int pa, int pb) {
  if (pa < 0 || pb < 0) return nullptr;
  bool a = false, b = false;
  for (int i = 0; i < ca.S; ++i) {
    a = a || ca.sel[i] == pa;
    b = b || ca.sel[i] == pb;
  }
  const auto it = h->pairing.find({pa, pb});
  return a && b && it != h->pairing.end() ? &it->second : nullptr;
}

// Forward passes with models pa and pb paired on one lane (each aligned pair of ops as
// one two-member launch, their other ops alone, in the merged order) and the other
// selected models one after another on a second lane, longest estimated alone time
// first.  Launches are enqueued alternating between the lanes.
static int forward_paired(rafiki_ensemble_t h, const CombineArgs& ca, const void* in, int n, hipStream_t s,
                          int pa, int pb, const std::vector<std::pair<int, int>>& steps, const CallScratch* ws) {
  std::vector<int> rest;
  for (int i = 0; i < ca.S; ++i)
    if (ca.sel[i] != pa && ca.sel[i] != pb) rest.push_back(ca.sel[i]);
  std::vector<double> est(h->n_models, 1.0);
  const auto mit = h->model_ms.find(n);
  if (mit != h->model_ms.end()) est = mit->second;
  std::stable_sort(rest.begin(), rest.end(), [&](int a, int b) { return est[a] > est[b]; });
  std::vector<std::pair<int, int>> lane_b;   // (model, op) in order
  for (int m : rest)
    for (size_t oi = 0; oi < h->models[m].ops.size(); ++oi) lane_b.push_back({m, (int)oi});
  Model& MA = h->models[pa];
  Model* MB = rest.empty() ? nullptr : &h->models[rest[0]];
  HIPCHK(hipEventRecord(h->staged_ev, s));
  HIPCHK(hipStreamWaitEvent(MA.stream, h->staged_ev, 0));
  if (MB) HIPCHK(hipStreamWaitEvent(MB->stream, h->staged_ev, 0));
  auto join = [&]() {
    hipError_t st = hipEventRecord(MA.done, MA.stream);
    if (st == hipSuccess) st = hipStreamWaitEvent(s, MA.done, 0);
    if (MB && st == hipSuccess) st = hipEventRecord(MB->done, MB->stream);
    if (MB && st == hipSuccess) st = hipStreamWaitEvent(s, MB->done, 0);
    return st;
  };
  float* lga = h->d_logits + (size_t)pa * ca.ld_model;
  float* lgb = h->d_logits + (size_t)pb * ca.ld_model;
  const size_t rounds = std::max(steps.size(), lane_b.size());
  for (size_t r = 0; r < rounds; ++r) {
    int rc = RAFIKI_OK;
    if (r < steps.size()) {
      const int i = steps[r].first, j = steps[r].second;
      if (i >= 0 && j >= 0) {
        const int mis[2] = {pa, pb}, ois[2] = {i, j};
        float* lg[2] = {lga, lgb};
        rc = run_op(h, mis, ois, 2, in, n, lg, MA.stream, ws);
      } else {
        const int mis[1] = {i >= 0 ? pa : pb}, ois[1] = {i >= 0 ? i : j};
        float* lg[1] = {i >= 0 ? lga : lgb};
        rc = run_op(h, mis, ois, 1, in, n, lg, MA.stream, ws);
      }
    }
    if (rc == RAFIKI_OK && r < lane_b.size()) {
      const int m = lane_b[r].first, oi = lane_b[r].second;
      rc = run_model(h, m, in, n, h->d_logits + (size_t)m * ca.ld_model, MB->stream, oi, oi + 1, ws);
    }
    if (rc) {
      (void)join();   // the caller's stream still waits for what the lanes already hold
      return rc;
    }
  }
  HIPCHK(join());
  return RAFIKI_OK;
}

static int forward(rafiki_ensemble_t h, const CombineArgs& ca, const void* in, int n, hipStream_t s,
                   rafiki_ensemble_s::Sched sched, const CallScratch* ws = nullptr) {
  const int solo = sched.solo;
  int rc = RAFIKI_OK;
  struct LeanScope {   // the schedule's tile tables for the launches enqueued below
    LeanScope(int level, int solo) { lean_tiles() = level; lean_gemm_model() = solo; }
    ~LeanScope() { lean_tiles() = 0; lean_gemm_model() = -1; }
  } lean_scope(sched.lean, sched.solo);
  if (fused_selection(h, ca)) {   // every selected model in one launch
    uint32_t mask = 0;
    for (int i = 0; i < ca.S; ++i) mask |= 1u << ca.sel[i];
    return run_fused(h, mask, in, n, h->d_logits, ca.ld_model, s);
  }
  if (grouped_selection(h, ca)) {   // one launch per op for up to kMaxGroup members, on the caller's stream
    for (int c0 = 0; c0 < ca.S; c0 += kMaxGroup) {
      const int nm = std::min(kMaxGroup, ca.S - c0);
      int mis[kMaxGroup];
      float* lg[kMaxGroup];
      for (int k = 0; k < nm; ++k) {
        mis[k] = ca.sel[c0 + k];
        lg[k] = h->d_logits + (size_t)mis[k] * ca.ld_model;
      }
      rc = run_models(h, mis, nm, in, n, lg, s, 0, SIZE_MAX, ws);
      if (rc) return rc;
    }
    return RAFIKI_OK;
  }
  const bool fork = h->concurrent && (!h->trace.on || h->trace.concurrent) && ca.S > 1;
  if (fork && sched.pa >= 0) {
    const auto* steps = selected_pairing(h, ca, sched.pa, sched.pb);
    if (steps) return forward_paired(h, ca, in, n, s, sched.pa, sched.pb, *steps, ws);
  }
  if (fork) {
    HIPCHK(hipEventRecord(h->staged_ev, s));
    // Lanes.  solo < 0: every model on its own lane.  solo = m: model m alone on one
    // lane, the other selected models one after another on a second lane, longest
    // (estimated alone) first, or shortest first if sched.ascending; each waits for
    // the previous one's done event.
    std::vector<int> prev(h->n_models, -1);        // model this one waits for (-1: staging)
    if (solo >= 0) {
      std::vector<double> est(h->n_models, 1.0);
      const auto it = h->model_ms.find(n);
      if (it != h->model_ms.end()) est = it->second;
      std::vector<int> rest;
      for (int i = 0; i < ca.S; ++i)
        if (ca.sel[i] != solo) rest.push_back(ca.sel[i]);
      std::stable_sort(rest.begin(), rest.end(), [&](int a, int b) { return est[a] > est[b]; });
      if (sched.ascending) std::reverse(rest.begin(), rest.end());
      for (size_t k = 1; k < rest.size(); ++k) prev[rest[k]] = rest[k - 1];
    }
    // enqueue offsets: a model's launches are enqueued after its predecessor's last one
    std::vector<size_t> off(h->n_models, 0);
    for (int i = 0; i < ca.S; ++i)           // a chain's predecessors come first in it
      for (int m = ca.sel[i]; prev[m] >= 0; m = prev[m]) off[ca.sel[i]] += h->models[prev[m]].ops.size();
    size_t rounds = 0;
    for (int i = 0; i < ca.S; ++i) {
      const int m = ca.sel[i];
      if (prev[m] < 0) HIPCHK(hipStreamWaitEvent(h->models[m].stream, h->staged_ev, 0));
      rounds = std::max(rounds, h->models[m].ops.size() + off[m]);
    }
    // On an error partway, the caller's stream still waits for whatever the model
    // streams already hold (they may read the caller's batch) before it is returned.
    auto join_after_error = [&](int code) {
      for (int i = 0; i < ca.S; ++i) {
        Model& M = h->models[ca.sel[i]];
        if (hipEventRecord(M.done, M.stream) == hipSuccess) (void)hipStreamWaitEvent(s, M.done, 0);
      }
      return code;
    };
    for (size_t r = 0; r < rounds; ++r)
      for (int i = 0; i < ca.S; ++i) {
        const int m = ca.sel[i];
        Model& M = h->models[m];
        if (r < off[m]) continue;
        const size_t oi = r - off[m];
        if (oi >= M.ops.size()) continue;
        hipError_t st = hipSuccess;
        if (oi == 0 && prev[m] >= 0) st = hipStreamWaitEvent(M.stream, h->models[prev[m]].done, 0);
        if (st != hipSuccess)
          return join_after_error(fail(RAFIKI_ERR_HIP, std::string("hipStreamWaitEvent: ") + hipGetErrorString(st)));
        rc = run_model(h, m, in, n, h->d_logits + (size_t)m * ca.ld_model, M.stream, oi, oi + 1, ws);
        if (rc) return join_after_error(rc);
        if (oi + 1 == M.ops.size()) st = hipEventRecord(M.done, M.stream);
        if (st != hipSuccess)
          return join_after_error(fail(RAFIKI_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(st)));
      }
    for (int i = 0; i < ca.S; ++i) HIPCHK(hipStreamWaitEvent(s, h->models[ca.sel[i]].done, 0));
  } else {
    for (int i = 0; i < ca.S; ++i) {
      const int m = ca.sel[i];
      rc = run_model(h, m, in, n, h->d_logits + (size_t)m * ca.ld_model, s, 0, SIZE_MAX, ws);
      if (rc) return rc;
    }
  }
  return RAFIKI_OK;
}

// The schedule of (n, mask): chosen on first use by timing every candidate on stream s
// (blocks the caller once).  Candidates: all models concurrent, and each selected model
// alone on one lane with the others chained on a second (longest first, and, with two
// or more chained, also shortest first).  A schedule only orders the same launches, so
// the choice never changes a result.  With fewer than three models, when tracing, or
// with model streams off, the models run as before (all concurrent).
static int pick_schedule(rafiki_ensemble_t h, const CombineArgs& ca, const void* in, int n, uint32_t mask,
                         hipStream_t s, rafiki_ensemble_s::Sched* sched, const CallScratch* ws = nullptr) {
  *sched = {};
  std::vector<std::pair<int, int>> pairs;   // pairable models of the selection
  for (const auto& kv : h->pairing)
    if (selected_pairing(h, ca, kv.first.first, kv.first.second)) pairs.push_back(kv.first);
  if ((ca.S < 3 && pairs.empty()) || !h->concurrent || (h->trace.on && !h->trace.concurrent) ||
      grouped_selection(h, ca) || fused_selection(h, ca))
    return RAFIKI_OK;
  const auto key = std::make_pair(n, mask);
  const auto it = h->schedule.find(key);
  if (it != h->schedule.end()) {
    *sched = it->second;
    return RAFIKI_OK;
  }
  if (!h->tune_schedule || h->trace.on) return RAFIKI_OK;   // never time candidates while tracing
  std::vector<rafiki_ensemble_s::Sched> cands(1);
  if (ca.S >= 3)
    for (int i = 0; i < ca.S; ++i) {
      cands.push_back({ca.sel[i], 0});
      cands.push_back({ca.sel[i], 1});
    }
  for (const auto& pr : pairs) cands.push_back({-1, 0, pr.first, pr.second});
  // each schedule also with the lean tiles, where they differ from the fastest alone
  const auto tl = h->tuned_lean.find(n), tf = h->tuned.find(n);
  bool differ = false;
  if (tl != h->tuned_lean.end() && tf != h->tuned.end())
    for (int i = 0; i < ca.S; ++i) differ = differ || tl->second[ca.sel[i]] != tf->second[ca.sel[i]];
  // and a schedule with a model alone on its lane also with that model's direct-conv
  // layers on GEMM tiles, where it has any
  const auto tg = h->tuned_lean_gemm.find(n);
  if (h->lean_policy && tl != h->tuned_lean.end() && tg != h->tuned_lean_gemm.end()) {
    const size_t k = cands.size();
    for (size_t i = 0; i < k; ++i) {
      rafiki_ensemble_s::Sched c = cands[i];
      if (differ) {
        c.lean = 1;
        cands.push_back(c);
      }
      if (c.solo >= 0 && tg->second[c.solo] != tl->second[c.solo]) {
        c.lean = 2;
        cands.push_back(c);
      }
    }
  }
  hipEvent_t ev[2] = {nullptr, nullptr};
  HIPCHK(hipEventCreate(&ev[0]));
  hipError_t st = hipEventCreate(&ev[1]);
  if (st != hipSuccess) {
    (void)hipEventDestroy(ev[0]);
    return fail(RAFIKI_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(st));
  }
  int rc = RAFIKI_OK;
  // Best of four runs each, the candidates taken in turn in every round, so that a drift
  // of the device's clocks during the timing affects them alike.
  std::vector<float> tbest(cands.size(), 1e30f);
  for (int rep = 0; rep < 4 && rc == RAFIKI_OK; ++rep)
    for (size_t ci = 0; ci < cands.size() && rc == RAFIKI_OK; ++ci) {
      st = hipEventRecord(ev[0], s);
      if (st == hipSuccess) rc = forward(h, ca, in, n, s, cands[ci], ws);
      if (st == hipSuccess && rc == RAFIKI_OK) st = hipEventRecord(ev[1], s);
      if (st == hipSuccess && rc == RAFIKI_OK) st = hipEventSynchronize(ev[1]);
      float ms = 0.f;
      if (st == hipSuccess && rc == RAFIKI_OK) st = hipEventElapsedTime(&ms, ev[0], ev[1]);
      if (st != hipSuccess && rc == RAFIKI_OK) rc = fail(RAFIKI_ERR_HIP, std::string("schedule timing: ") + hipGetErrorString(st));
      if (rc == RAFIKI_OK) tbest[ci] = std::min(tbest[ci], ms);
    }
  rafiki_ensemble_s::Sched best_sched;
  float best = 1e30f;
  for (size_t ci = 0; ci < cands.size() && rc == RAFIKI_OK; ++ci)
    if (tbest[ci] < best) { best = tbest[ci]; best_sched = cands[ci]; }
  (void)hipEventDestroy(ev[0]);
  (void)hipEventDestroy(ev[1]);
  if (rc) return rc;
  h->schedule[key] = best_sched;
  *sched = best_sched;
  return RAFIKI_OK;
}

constexpr size_t kMaxGraphs = 64;   // (batch size, subset) pairs kept as graphs per handle

// The instantiated graph of the forward passes for (n, mask), captured on first use.
// *exec stays null when the cache is full or the capture fails; the caller then runs
// the same launches eagerly (a failed capture is counted and disables graphs).
static int graph_for(rafiki_ensemble_t h, int n, uint32_t mask, const CombineArgs& ca, const void* in,
                     rafiki_ensemble_s::Sched sched, hipGraphExec_t* exec) {
  *exec = nullptr;
  const auto key = std::make_pair(n, mask);
  const auto it = h->graphs.find(key);
  if (it != h->graphs.end()) {
    *exec = it->second.exec;
    return RAFIKI_OK;
  }
  if (h->graphs.size() >= kMaxGraphs) return RAFIKI_OK;
  hipStream_t cs = h->capture_stream;
  if (hipStreamBeginCapture(cs, hipStreamCaptureModeRelaxed) != hipSuccess) {
    (void)hipGetLastError();
    ++h->graph_failures;
    h->use_graphs = false;
    return RAFIKI_OK;
  }
  const int frc = forward(h, ca, in, n, cs, sched);
  hipGraph_t g = nullptr;
  const hipError_t est = hipStreamEndCapture(cs, &g);
  hipGraphExec_t x = nullptr;
  hipError_t ist = hipErrorUnknown;
  if (frc == RAFIKI_OK && est == hipSuccess && g) ist = hipGraphInstantiate(&x, g, nullptr, nullptr, 0);
  if (frc != RAFIKI_OK || est != hipSuccess || ist != hipSuccess) {
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();
    ++h->graph_failures;
    h->use_graphs = false;
    return RAFIKI_OK;
  }
  h->graphs[key] = {g, x};
  *exec = x;
  return RAFIKI_OK;
}

// One scheduled batch through the selected models, then the mean (vote = false) or
// majority-vote (vote = true) combine into out / out_labels.
static int serve(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask, float* out,
                 int32_t* out_labels, void* stream, bool vote, const CallScratch* ws = nullptr) {
  int rc = check_call(h, batch, n);
  if (rc) return rc;
  if (!out || !out_labels) return fail(RAFIKI_ERR_INVALID, "null output pointer");
  if (model_subset_mask == 0) return fail(RAFIKI_ERR_INVALID, "model_subset_mask must select at least one model");
  if (h->n_models < 32 && (model_subset_mask >> h->n_models) != 0)
    return fail(RAFIKI_ERR_INVALID, "model_subset_mask selects a model that does not exist");
  hipStream_t s = (hipStream_t)stream;
  CombineArgs ca{};
  ca.logits = h->d_logits;
  ca.ld_model = (long long)h->max_batch * h->n_classes;
  ca.n = n; ca.C = h->n_classes; ca.probs = out; ca.labels = out_labels;
  for (int m = 0; m < h->n_models; ++m)
    if ((model_subset_mask >> m) & 1u) ca.sel[ca.S++] = m;
  // With graphs on, a graph replays the forward passes once this batch size is tuned;
  // tracing, and a batch size seen for the first time, run them eagerly.
  const bool graph = h->use_graphs && !h->trace.on && h->tuned.count(n) && !ws;
  if (graph) {
    const void* in = h->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32 ? h->d_staged : h->d_tokens;
    rc = stage(h, batch, n, s, h->d_staged);
    if (rc) return rc;
    if (h->input_kind == RAFIKI_INPUT_TOKENS_I32)
      HIPCHK(hipMemcpyAsync(h->d_tokens, batch, (size_t)n * h->H * 4, hipMemcpyDeviceToDevice, s));
    hipGraphExec_t exec = nullptr;
    rafiki_ensemble_s::Sched sched;
    rc = pick_schedule(h, ca, in, n, model_subset_mask, s, &sched);
    if (rc) return rc;
    rc = graph_for(h, n, model_subset_mask, ca, in, sched, &exec);
    if (rc) return rc;
    if (exec) {
      HIPCHK(hipGraphLaunch(exec, s));
      ++h->graph_replays;
    } else {
      rc = forward(h, ca, in, n, s, sched);   // capture refused: the same launches, eagerly
      if (rc) return rc;
    }
  } else {
    const void* in = model_input(h, batch, h->d_staged);
    rc = stage(h, batch, n, s, h->d_staged);
    if (!rc) rc = tune(h, n, in, s);
    rafiki_ensemble_s::Sched sched;
    if (!rc) rc = pick_schedule(h, ca, in, n, model_subset_mask, s, &sched, ws);
    if (!rc) rc = forward(h, ca, in, n, s, sched, ws);
    if (rc) return rc;
  }
  const double cbytes = (double)n * h->n_classes * 4.0 * (ca.S + 1) + 4.0 * n;
  if (vote) {
    TRACED(h, s, RAFIKI_K_VOTE, -1, -1, 0.0, cbytes, launch_vote(ca, s));
  } else {
    TRACED(h, s, RAFIKI_K_COMBINE, -1, -1, 0.0, cbytes, launch_combine(ca, s));
  }
  return RAFIKI_OK;
}

extern "C" {

int rafiki_ensemble_infer(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                          float* out_probs, int32_t* out_labels, void* stream) {
  return serve(h, batch, n, model_subset_mask, out_probs, out_labels, stream, false);
}

int rafiki_ensemble_infer_vote(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                               float* out_votes, int32_t* out_labels, void* stream) {
  return serve(h, batch, n, model_subset_mask, out_votes, out_labels, stream, true);
}

int rafiki_ensemble_infer_noalloc(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                                  float* out_probs, int32_t* out_labels, void* stream) {
  int rc = check_call(h, batch, n);
  if (rc) return rc;
  if (model_subset_mask == 0) return fail(RAFIKI_ERR_INVALID, "model_subset_mask must select at least one model");
  if (h->n_models < 32 && (model_subset_mask >> h->n_models) != 0)
    return fail(RAFIKI_ERR_INVALID, "model_subset_mask selects a model that does not exist");
  if (!h->scratch) return fail(RAFIKI_ERR_HIP, "no-alloc scratch unavailable: " + h->scratch_err);
  // Layout for this call: every selected model's epilogue-max keys first (one range,
  // cleared below), then each model's split-K partial sums, 256-byte aligned.
  CallScratch ws;
  char* base = (char*)h->scratch;
  size_t off = 0;
  for (int m = 0; m < h->n_models; ++m) {
    if (!((model_subset_mask >> m) & 1u)) continue;
    ws.slot[m] = (unsigned*)(base + off);
    for (const Op& op : h->models[m].ops)
      if (op.d_slot) off += (size_t)n * op.ldslot * 4;
    off = round_up_sz(off, 256);
  }
  const size_t slot_bytes = off;
  for (int m = 0; m < h->n_models; ++m) {
    if (!((model_subset_mask >> m) & 1u) || h->precision != RAFIKI_BF16) continue;
    size_t need = 0;
    for (const Op& op : h->models[m].ops) {
      if (op.kind != O_CONV && op.kind != O_CONV1D) continue;
      const int rows = n * op.Ho * op.Wo;
      const int sp = choose_splits(rows, op.c_out, op.Kp / 64);
      if (sp > 1) need = std::max(need, (size_t)sp * rows * op.Co_pad * 4);
    }
    ws.partial[m] = (float*)(base + off);
    ws.partial_bytes[m] = need;
    off = round_up_sz(off + need, 256);
  }
  if (off > kNoAllocScratchBytes)
    return fail(RAFIKI_ERR_UNSUPPORTED, "this call needs " + std::to_string(off) + " bytes of scratch; the no-alloc "
                "scratch holds " + std::to_string(kNoAllocScratchBytes) + " (use a smaller n or fewer models, or infer)");
  hipStream_t s = (hipStream_t)stream;
  if (slot_bytes) {   // the maxima start from the zero key; the array keeps the last call's contents
    const long long words = (long long)(slot_bytes / 4);
    launch(zero_u32_kernel, dim3((unsigned)((words + 255) / 256)), dim3(256), s, (unsigned*)base, words);
    HIPCHK(hipGetLastError());
  }
  return serve(h, batch, n, model_subset_mask, out_probs, out_labels, stream, false, &ws);
}

int rafiki_ensemble_model_logits(rafiki_ensemble_t h, int model, const void* batch, int n, float* out_logits,
                                 void* stream) {
  int rc = check_call(h, batch, n);
  if (rc) return rc;
  if (!out_logits) return fail(RAFIKI_ERR_INVALID, "null output pointer");
  if (model < 0 || model >= h->n_models) return fail(RAFIKI_ERR_INVALID, "model index out of range");
  hipStream_t s = (hipStream_t)stream;
  const void* in = model_input(h, batch, h->d_staged);
  rc = stage(h, batch, n, s, h->d_staged);
  if (rc) return rc;
  if (fused_model(h, model)) return run_fused(h, 1u << model, in, n, out_logits, 0, s);
  rc = tune(h, n, in, s);
  if (rc) return rc;
  return run_model(h, model, in, n, out_logits, s);
}

int rafiki_ensemble_info(rafiki_ensemble_t h, int* n_models, int* n_classes, int* max_batch) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (n_models) *n_models = h->n_models;
  if (n_classes) *n_classes = h->n_classes;
  if (max_batch) *max_batch = h->max_batch;
  return RAFIKI_OK;
}

int rafiki_ensemble_destroy(rafiki_ensemble_t h) {
  if (!h) return RAFIKI_OK;
  hipError_t st = hipDeviceSynchronize();
  delete h;
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipDeviceSynchronize: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_ensemble_trace(rafiki_ensemble_t h, int enable) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (enable < 0 || enable > 2) return fail(RAFIKI_ERR_INVALID, "trace mode must be 0, 1 or 2");
  h->trace.on = enable != 0;
  h->trace.concurrent = enable == 2;
  h->trace.recs.clear();
  h->trace.used = 0;
  return RAFIKI_OK;
}

int rafiki_ensemble_trace_read(rafiki_ensemble_t h, rafiki_trace_rec* out, int cap, int* count) {
  if (!h || !count || (cap > 0 && !out)) return fail(RAFIKI_ERR_INVALID, "null argument");
  const int total = (int)h->trace.recs.size();
  *count = total;
  if (cap < total) return RAFIKI_OK;   // too small: keep the records, report the count
  for (int i = 0; i < total; ++i) {
    const auto& r = h->trace.recs[i];
    hipError_t st = hipEventSynchronize(r.b);
    if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipEventSynchronize: ") + hipGetErrorString(st));
    float ms = 0.f;
    st = hipEventElapsedTime(&ms, r.a, r.b);
    if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipEventElapsedTime: ") + hipGetErrorString(st));
    out[i].kind = r.kind; out[i].model = r.model; out[i].layer = r.layer;
    out[i].flops = r.flops; out[i].bytes = r.bytes; out[i].ms = ms;
    out[i].tile_cfg = r.tile_cfg; out[i].splits = r.splits;
  }
  h->trace.recs.clear();
  h->trace.used = 0;
  return RAFIKI_OK;
}

static int combine_standalone(const float* logits, int n_models, int n, int n_classes, float* out,
                              int32_t* labels, void* stream, bool vote) {
  if (!logits || !out || !labels) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (n_models < 1 || n_models > 32) return fail(RAFIKI_ERR_INVALID, "n_models must be in [1, 32]");
  if (n < 1 || n_classes < 1 || n_classes > 1024)
    return fail(RAFIKI_ERR_INVALID, "n must be >= 1 and n_classes in [1, 1024]");
  CombineArgs ca{};
  ca.logits = logits;
  ca.ld_model = (long long)n * n_classes;
  for (int m = 0; m < n_models; ++m) ca.sel[ca.S++] = m;
  ca.n = n; ca.C = n_classes; ca.probs = out; ca.labels = labels;
  const hipError_t st = vote ? launch_vote(ca, (hipStream_t)stream) : launch_combine(ca, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("combine launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_combine_mean(const float* logits, int n_models, int n, int n_classes, float* out_probs,
                        int32_t* out_labels, void* stream) {
  return combine_standalone(logits, n_models, n, n_classes, out_probs, out_labels, stream, false);
}

int rafiki_combine_vote(const float* logits, int n_models, int n, int n_classes, float* out_votes,
                        int32_t* out_labels, void* stream) {
  return combine_standalone(logits, n_models, n, n_classes, out_votes, out_labels, stream, true);
}

int rafiki_maxpool_nhwc_bf16(const void* x, void* y, int n, int h, int w, int c, int k, int stride, int pad,
                             void* stream) {
  if (!x || !y) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (n < 1 || h < 1 || w < 1 || c < 8 || c % 8 || k < 1 || stride < 1 || pad < 0 || pad >= k)
    return fail(RAFIKI_ERR_INVALID, "maxpool geometry invalid (c a multiple of 8, pad < k)");
  if (h + 2 * pad < k || w + 2 * pad < k) return fail(RAFIKI_ERR_INVALID, "maxpool output would be empty");
  const int ho = (h + 2 * pad - k) / stride + 1, wo = (w + 2 * pad - k) / stride + 1;
  const hipError_t st = launch_maxpool(x, y, n, h, w, c, ho, wo, k, stride, pad, 1, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("maxpool launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_global_avgpool_nhwc_bf16(const void* x, void* y, int n, int h, int w, int c, void* stream) {
  if (!x || !y) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (n < 1 || h < 1 || w < 1 || c < 8 || c % 8) return fail(RAFIKI_ERR_INVALID, "pool geometry invalid");
  const hipError_t st = launch_spatial_reduce(x, y, n, h * w, c, 0, 1, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("pool launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_probe_mfma_bf16(int blocks, int iters, float* out, void* stream) {
  if (!out) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (blocks < 1 || iters < 1) return fail(RAFIKI_ERR_INVALID, "blocks and iters must be positive");
  const hipError_t st = launch_probe_mfma(blocks, iters, out, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("probe launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_probe_hbm_read(const void* x, long long bytes, int blocks, unsigned* out, void* stream) {
  if (!x || !out) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (bytes < 16 || bytes % 16 || ((uintptr_t)x & 15) || blocks < 1)
    return fail(RAFIKI_ERR_INVALID, "bytes must be a positive multiple of 16, x 16-byte aligned, blocks >= 1");
  const hipError_t st = launch_probe_read(x, bytes / 16, blocks, out, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("probe launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_probe_mainloop(int variant, int sync, int blocks, int ktiles, float* out, void* stream) {
  if (!out) return fail(RAFIKI_ERR_INVALID, "null pointer");
  if (variant < 0 || variant > 3) return fail(RAFIKI_ERR_INVALID, "variant must be 0..3");
  if (blocks < 1 || ktiles < 1) return fail(RAFIKI_ERR_INVALID, "blocks and ktiles must be positive");
  const hipError_t st = launch_probe_mainloop(variant, sync != 0, blocks, ktiles, out, (hipStream_t)stream);
  if (st != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("probe launch: ") + hipGetErrorString(st));
  return RAFIKI_OK;
}

int rafiki_tile_config(int cfg, int* bm, int* bn, int* waves, int* stages, int* bk) {
  if (cfg < 0 || cfg >= kNumMfmaConfigs) return fail(RAFIKI_ERR_INVALID, "no such tile configuration");
  const MfmaConfig& c = kMfmaConfigs[cfg];
  if (bm) *bm = c.bm;
  if (bn) *bn = c.bn;
  if (waves) *waves = c.waves;
  if (stages) *stages = c.stages;
  if (bk) *bk = c.bk;
  return RAFIKI_OK;
}

int rafiki_ensemble_force_tile(rafiki_ensemble_t h, int cfg) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (cfg == RAFIKI_TILE_DIRECT) cfg = kCfgDirect;
  else if (cfg < -1 || cfg >= kNumMfmaConfigs) return fail(RAFIKI_ERR_INVALID, "no such tile configuration");
  if (cfg != h->force_tile) {
    HIPCHK(hipDeviceSynchronize());   // graphs holding the old tiles may still be running
    h->drop_graphs();
  }
  h->force_tile = cfg;
  return RAFIKI_OK;
}

int rafiki_ensemble_get_schedule(rafiki_ensemble_t h, int n, uint32_t mask, int* solo, int* ascending) {
  if (!h || !solo) return fail(RAFIKI_ERR_INVALID, "null argument");
  const auto it = h->schedule.find(std::make_pair(n, mask));
  if (it == h->schedule.end()) return fail(RAFIKI_ERR_INVALID, "no schedule chosen for this batch size and subset");
  *solo = it->second.solo;
  if (ascending) *ascending = it->second.ascending;
  return RAFIKI_OK;
}

int rafiki_ensemble_set_schedule(rafiki_ensemble_t h, int n, uint32_t mask, int solo, int ascending) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (n < 1 || n > h->max_batch || mask == 0 || (h->n_models < 32 && (mask >> h->n_models) != 0))
    return fail(RAFIKI_ERR_INVALID, "batch size or subset mask out of range");
  if (solo < -1 || solo >= h->n_models || (solo >= 0 && !((mask >> solo) & 1u)))
    return fail(RAFIKI_ERR_INVALID, "solo must be -1 or a model of the subset");
  HIPCHK(hipDeviceSynchronize());   // graphs built with the old schedule may still run
  h->drop_graphs();
  h->schedule[std::make_pair(n, mask)] = {solo, ascending ? 1 : 0};
  return RAFIKI_OK;
}

int rafiki_ensemble_get_schedule_tiles(rafiki_ensemble_t h, int n, uint32_t mask, int* lean) {
  if (!h || !lean) return fail(RAFIKI_ERR_INVALID, "null argument");
  const auto it = h->schedule.find(std::make_pair(n, mask));
  if (it == h->schedule.end()) return fail(RAFIKI_ERR_INVALID, "no schedule chosen for this batch size and subset");
  *lean = it->second.lean;
  return RAFIKI_OK;
}

int rafiki_ensemble_set_schedule_tiles(rafiki_ensemble_t h, int n, uint32_t mask, int lean) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (lean < 0 || lean > 2) return fail(RAFIKI_ERR_INVALID, "lean must be 0, 1 or 2");
  const auto it = h->schedule.find(std::make_pair(n, mask));
  if (it == h->schedule.end()) return fail(RAFIKI_ERR_INVALID, "no schedule chosen for this batch size and subset");
  HIPCHK(hipDeviceSynchronize());   // graphs built with the old policy may still run
  h->drop_graphs();
  it->second.lean = lean;
  return RAFIKI_OK;
}

int rafiki_ensemble_get_schedule_pair(rafiki_ensemble_t h, int n, uint32_t mask, int* pa, int* pb) {
  if (!h || !pa || !pb) return fail(RAFIKI_ERR_INVALID, "null argument");
  const auto it = h->schedule.find(std::make_pair(n, mask));
  if (it == h->schedule.end()) return fail(RAFIKI_ERR_INVALID, "no schedule chosen for this batch size and subset");
  *pa = it->second.pa;
  *pb = it->second.pb;
  return RAFIKI_OK;
}

int rafiki_ensemble_set_schedule_pair(rafiki_ensemble_t h, int n, uint32_t mask, int pa, int pb) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (n < 1 || n > h->max_batch || mask == 0 || (h->n_models < 32 && (mask >> h->n_models) != 0))
    return fail(RAFIKI_ERR_INVALID, "batch size or subset mask out of range");
  if (pa != -1 && (pa < 0 || pb <= pa || pb >= h->n_models || !((mask >> pa) & 1u) || !((mask >> pb) & 1u) ||
                   !h->pairing.count({pa, pb})))
    return fail(RAFIKI_ERR_INVALID, "pa < pb must be a pairable pair of the subset, or pa = -1");
  HIPCHK(hipDeviceSynchronize());   // graphs built with the old schedule may still run
  h->drop_graphs();
  rafiki_ensemble_s::Sched sc;
  if (pa >= 0) {
    sc.pa = pa;
    sc.pb = pb;
  }
  h->schedule[std::make_pair(n, mask)] = sc;
  return RAFIKI_OK;
}

int rafiki_ensemble_pairing(rafiki_ensemble_t h, int a, int b, int* aligned) {
  if (!h || !aligned) return fail(RAFIKI_ERR_INVALID, "null argument");
  if (a < 0 || b <= a || b >= h->n_models) return fail(RAFIKI_ERR_INVALID, "need 0 <= a < b < n_models");
  *aligned = 0;
  const auto it = h->pairing.find({a, b});
  if (it != h->pairing.end())
    for (const auto& st : it->second) *aligned += st.first >= 0 && st.second >= 0;
  return RAFIKI_OK;
}

int rafiki_ensemble_use_graphs(rafiki_ensemble_t h, int enable) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  HIPCHK(hipDeviceSynchronize());
  h->drop_graphs();
  h->use_graphs = enable != 0;
  return RAFIKI_OK;
}

int rafiki_ensemble_graph_stats(rafiki_ensemble_t h, int* n_graphs, long long* replays, long long* failures) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (n_graphs) *n_graphs = (int)h->graphs.size();
  if (replays) *replays = h->graph_replays;
  if (failures) *failures = h->graph_failures;
  return RAFIKI_OK;
}

const char* rafiki_last_error(void) { return g_err.c_str(); }

}  // extern "C"

// ---------------------------------------------------------------- serving
namespace {

using SteadyClock = std::chrono::steady_clock;

// Microseconds since construction; waits sleep coarsely, then spin for the last
// few hundred microseconds.
struct ServeClock {
  SteadyClock::time_point t0 = SteadyClock::now();
  int64_t now() const {
    return std::chrono::duration_cast<std::chrono::microseconds>(SteadyClock::now() - t0).count();
  }
  void wait_until(int64_t t) const {
    for (;;) {
      const int64_t d = t - now();
      if (d <= 0) return;
      if (d > 400) std::this_thread::sleep_for(std::chrono::microseconds(d - 300));
      else std::this_thread::yield();
    }
  }
};

int64_t cost_of(const rafiki_greedy_policy& p, int32_t b) {
  for (int i = 0; i < p.n_sizes; ++i)
    if (p.batch_sizes[i] == b) return p.cost_us[i];
  return 0;
}

size_t request_bytes(const rafiki_ensemble_s* h) { return (size_t)h->C * h->H * h->W * 4; }

const void* request_row(const rafiki_ensemble_s* h, const void* requests, int64_t i) {
  return (const char*)requests + (size_t)i * request_bytes(h);
}

int check_mask(const rafiki_ensemble_s* h, uint32_t mask) {
  if (mask == 0) return fail(RAFIKI_ERR_INVALID, "model_subset_mask must select at least one model");
  if (h->n_models < 32 && (mask >> h->n_models) != 0)
    return fail(RAFIKI_ERR_INVALID, "model_subset_mask selects a model that does not exist");
  return RAFIKI_OK;
}

int check_serve_outputs(const void* requests, int64_t n, float* probs, int32_t* labels, int64_t* lat,
                        rafiki_dispatch* disp, int64_t cap, int64_t* ndisp) {
  if (n > 0 && (!requests || !probs || !labels || !lat))
    return fail(RAFIKI_ERR_INVALID, "null request or output pointer");
  if (!ndisp || cap < 0 || (cap > 0 && !disp)) return fail(RAFIKI_ERR_INVALID, "null dispatch output or negative cap");
  if (n > (int64_t)INT32_MAX) return fail(RAFIKI_ERR_INVALID, "too many requests");
  return RAFIKI_OK;
}

int check_policy_fits(const rafiki_ensemble_s* h, const rafiki_greedy_policy* p) {
  int rc = check_policy(p);
  if (rc) return rc;
  if (p->batch_sizes[p->n_sizes - 1] > h->max_batch)
    return fail(RAFIKI_ERR_INVALID, "the largest batch size exceeds max_batch");
  return RAFIKI_OK;
}

void record(rafiki_dispatch* disp, int64_t cap, int64_t& nd, const rafiki_dispatch& d) {
  if (nd < cap) disp[nd] = d;
  ++nd;
}

// One model's whole pipeline for asynchronous serving on its own stream: stage into
// its own buffer, forward pass, softmax + argmax of its logits into the output rows.
int launch_single(rafiki_ensemble_s* h, int m, const void* rows, int b, float* probs, int32_t* labels) {
  Model& M = h->models[m];
  const void* in = model_input(h, rows, M.d_staged_own);
  int rc = stage(h, rows, b, M.stream, M.d_staged_own);
  if (rc) return rc;
  float* logits = h->d_logits + (size_t)m * h->max_batch * h->n_classes;
  rc = run_model(h, m, in, b, logits, M.stream);
  if (rc) return rc;
  CombineArgs ca{};
  ca.logits = logits;
  ca.ld_model = 0;
  ca.sel[0] = 0;
  ca.S = 1;
  ca.n = b; ca.C = h->n_classes; ca.probs = probs; ca.labels = labels;
  HIPCHK(launch_combine(ca, M.stream));
  HIPCHK(hipEventRecord(M.done, M.stream));
  return RAFIKI_OK;
}

}  // namespace

extern "C" {

int rafiki_ensemble_profile(rafiki_ensemble_t h, const void* batch, const int32_t* batch_sizes, int n_sizes,
                            uint32_t mask, int reps, float* scratch_probs, int32_t* scratch_labels,
                            int64_t* out_cost_us, void* stream) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (!batch || !batch_sizes || !scratch_probs || !scratch_labels || !out_cost_us)
    return fail(RAFIKI_ERR_INVALID, "null argument");
  if (n_sizes < 1 || n_sizes > 64 || reps < 1 || reps > 1000)
    return fail(RAFIKI_ERR_INVALID, "n_sizes must be in [1, 64] and reps in [1, 1000]");
  for (int i = 0; i < n_sizes; ++i)
    if (batch_sizes[i] < 1 || batch_sizes[i] > h->max_batch)
      return fail(RAFIKI_ERR_INVALID, "batch sizes must be in [1, max_batch]");
  int rc = check_mask(h, mask);
  if (rc) return rc;
  hipStream_t s = (hipStream_t)stream;
  hipEvent_t ev[2] = {nullptr, nullptr};
  HIPCHK(hipEventCreate(&ev[0]));
  if (hipEventCreate(&ev[1]) != hipSuccess) {
    (void)hipEventDestroy(ev[0]);
    return fail(RAFIKI_ERR_HIP, "hipEventCreate failed");
  }
  std::vector<float> t(reps);
  for (int i = 0; i < n_sizes && !rc; ++i) {
    const int b = batch_sizes[i];
    rc = serve(h, batch, b, mask, scratch_probs, scratch_labels, stream, false);   // untimed (tunes b)
    for (int r = 0; r < reps && !rc; ++r) {
      if (hipEventRecord(ev[0], s) != hipSuccess) { rc = fail(RAFIKI_ERR_HIP, "hipEventRecord failed"); break; }
      rc = serve(h, batch, b, mask, scratch_probs, scratch_labels, stream, false);
      if (rc) break;
      if (hipEventRecord(ev[1], s) != hipSuccess || hipEventSynchronize(ev[1]) != hipSuccess ||
          hipEventElapsedTime(&t[r], ev[0], ev[1]) != hipSuccess)
        rc = fail(RAFIKI_ERR_HIP, "event timing failed");
    }
    if (rc) break;
    std::sort(t.begin(), t.end());
    out_cost_us[i] = (int64_t)std::ceil((double)t[reps / 2] * 1000.0);
  }
  (void)hipEventDestroy(ev[0]);
  (void)hipEventDestroy(ev[1]);
  return rc;
}

int rafiki_ensemble_serve_greedy(rafiki_ensemble_t h, const void* requests, const int64_t* arrival_us,
                                 int64_t n_requests, const rafiki_greedy_policy* policy, uint32_t mask,
                                 int combine, float* out_probs, int32_t* out_labels, int64_t* out_latency_us,
                                 rafiki_dispatch* out_dispatch, int64_t dispatch_cap, int64_t* out_n_dispatch,
                                 void* stream) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  int rc = check_policy_fits(h, policy);
  if (!rc) rc = check_arrivals(arrival_us, n_requests);
  if (!rc) rc = check_mask(h, mask);
  if (!rc) rc = check_serve_outputs(requests, n_requests, out_probs, out_labels, out_latency_us, out_dispatch,
                                    dispatch_cap, out_n_dispatch);
  if (rc) return rc;
  if (combine != 0 && combine != 1) return fail(RAFIKI_ERR_INVALID, "combine must be 0 (mean) or 1 (vote)");
  const rafiki_greedy_policy& p = *policy;
  const bool vote = combine == 1;
  const int64_t n = n_requests;
  const int C = h->n_classes;
  hipStream_t s = (hipStream_t)stream;
  std::fill(out_latency_us, out_latency_us + n, int64_t(-1));
  *out_n_dispatch = 0;
  // Warm up (and tune) every candidate size before the clock starts.
  for (int i = 0; i < p.n_sizes; ++i) {
    const int b = p.batch_sizes[i];
    if (b > n) break;
    rc = serve(h, requests, b, mask, out_probs, out_labels, stream, vote);
    if (rc) return rc;
  }
  HIPCHK(hipStreamSynchronize(s));
  int64_t nd = 0, head = 0, arrived = 0;
  const int64_t* a = arrival_us;
  ServeClock clk;
  while (head < n) {
    const int64_t t = clk.now();
    while (arrived < n && a[arrived] <= t) ++arrived;
    const int64_t qlen = arrived - head;
    if (qlen == 0) {
      clk.wait_until(a[arrived]);
      continue;
    }
    const int64_t wait = t - a[head];
    const int32_t b = greedy_decide(p, qlen, wait);
    if (b > 0) {
      rc = serve(h, request_row(h, requests, head), b, mask, out_probs + (size_t)head * C, out_labels + head,
                 stream, vote);
      if (rc) return rc;
      HIPCHK(hipStreamSynchronize(s));
      const int64_t done = clk.now();
      for (int64_t i = head; i < head + b; ++i) out_latency_us[i] = done - a[i];
      record(out_dispatch, dispatch_cap, nd, {t, done, head, qlen, wait, b, -1});
      head += b;
      continue;
    }
    int64_t next = arrived < n ? a[arrived] : INT64_MAX;
    next = std::min(next, greedy_deadline(p, qlen, a[head]));
    if (next == INT64_MAX) break;   // fewer than min(B) left, nothing more arriving
    clk.wait_until(next);
  }
  *out_n_dispatch = nd;
  return RAFIKI_OK;
}

int rafiki_ensemble_serve_rl(rafiki_ensemble_t h, rafiki_rl_t agent, const void* requests, const int64_t* arrival_us,
                             int64_t n_requests, int mode, uint64_t seed, float* out_probs, int32_t* out_labels,
                             int64_t* out_latency_us, rafiki_dispatch* out_dispatch, int32_t* out_actions,
                             double* out_states, int64_t cap, int64_t* out_steps, void* stream) {
  if (!h || !agent) return fail(RAFIKI_ERR_INVALID, "null handle or agent");
  if (mode != 1 && mode != 2) return fail(RAFIKI_ERR_INVALID, "mode must be 1 (sample) or 2 (most probable)");
  int rc = check_arrivals(arrival_us, n_requests);
  if (!rc) rc = check_serve_outputs(requests, n_requests, out_probs, out_labels, out_latency_us, out_dispatch, cap,
                                    out_steps);
  if (rc) return rc;
  if (cap > 0 && (!out_actions || !out_states)) return fail(RAFIKI_ERR_INVALID, "null action or state log");
  const RlAgentView ag = rl_view(agent);
  if (ag.n_models != h->n_models) return fail(RAFIKI_ERR_INVALID, "the agent schedules a different number of models");
  if (ag.batch_sizes[ag.n_sizes - 1] > h->max_batch)
    return fail(RAFIKI_ERR_INVALID, "the agent's largest batch size exceeds max_batch");
  const int64_t n = n_requests;
  const int C = h->n_classes;
  hipStream_t s = (hipStream_t)stream;
  std::fill(out_latency_us, out_latency_us + n, int64_t(-1));
  *out_steps = 0;
  // Warm up (and tune) every subset at every size a batch can take -- min(b, queue
  // length) is any of 1 .. max(B) -- before the clock starts.
  for (int b = 1; b <= ag.batch_sizes[ag.n_sizes - 1] && b <= n; ++b)
    for (int v = 1; v < (1 << h->n_models); ++v) {
      rc = serve(h, requests, b, (uint32_t)v, out_probs, out_labels, stream, false);
      if (rc) return rc;
    }
  HIPCHK(hipStreamSynchronize(s));
  std::vector<double> state(ag.state_dim);
  std::vector<int64_t> waits((size_t)ag.queue_features), busy_left(h->n_models, 0);
  uint64_t rng = seed;
  int64_t k = 0, head = 0, arrived = 0;
  const int64_t* a = arrival_us;
  ServeClock clk;
  while (head < n) {
    const int64_t t = clk.now();
    while (arrived < n && a[arrived] <= t) ++arrived;
    const int64_t qlen = arrived - head;
    if (qlen == 0) {
      clk.wait_until(a[arrived]);
      continue;
    }
    // Every model is free here: the previous batch has completed on the device.
    const int64_t nq = std::min<int64_t>(qlen, ag.queue_features);
    for (int64_t i = 0; i < nq; ++i) waits[i] = t - a[head + i];
    rl_live_state(agent, waits.data(), nq, busy_left.data(), state.data());
    const int act = rl_choose(agent, state.data(), mode, &rng);
    int mask = 0, j = 0;
    rl_action(agent, act, &mask, &j);
    const int b = (int)std::min<int64_t>(ag.batch_sizes[j], qlen);
    rc = serve(h, request_row(h, requests, head), b, (uint32_t)mask, out_probs + (size_t)head * C, out_labels + head,
               stream, false);
    if (rc) return rc;
    HIPCHK(hipStreamSynchronize(s));
    const int64_t done = clk.now();
    for (int64_t i = head; i < head + b; ++i) out_latency_us[i] = done - a[i];
    if (k < cap) {
      out_dispatch[k] = {t, done, head, qlen, t - a[head], b, -1};
      out_actions[k] = act;
      std::copy(state.begin(), state.end(), out_states + (size_t)k * ag.state_dim);
    }
    ++k;
    head += b;
  }
  *out_steps = k;
  return RAFIKI_OK;
}

int rafiki_ensemble_serve_greedy_async(rafiki_ensemble_t h, const void* requests, const int64_t* arrival_us,
                                       int64_t n_requests, const rafiki_greedy_policy* policies, uint32_t mask,
                                       float* out_probs, int32_t* out_labels, int64_t* out_latency_us,
                                       rafiki_dispatch* out_dispatch, int64_t dispatch_cap, int64_t* out_n_dispatch,
                                       void* stream) {
  if (!h) return fail(RAFIKI_ERR_INVALID, "null handle");
  if (!policies) return fail(RAFIKI_ERR_INVALID, "null policies");
  int rc = check_mask(h, mask);
  if (!rc) rc = check_arrivals(arrival_us, n_requests);
  if (!rc) rc = check_serve_outputs(requests, n_requests, out_probs, out_labels, out_latency_us, out_dispatch,
                                    dispatch_cap, out_n_dispatch);
  if (rc) return rc;
  std::vector<int> sel;
  for (int m = 0; m < h->n_models; ++m)
    if ((mask >> m) & 1u) {
      rc = check_policy_fits(h, &policies[m]);
      if (rc) return rc;
      sel.push_back(m);
    }
  const int64_t n = n_requests;
  const int C = h->n_classes;
  std::fill(out_latency_us, out_latency_us + n, int64_t(-1));
  *out_n_dispatch = 0;
  HIPCHK(hipStreamSynchronize((hipStream_t)stream));   // requests written on the caller's stream
  if (h->input_kind == RAFIKI_INPUT_IMAGE_NCHW_F32)
    for (int m : sel)
      if (!h->models[m].d_staged_own) {
        rc = dev_alloc(h, &h->models[m].d_staged_own,
                       (size_t)h->max_batch * h->H * h->W * h->in_Cs * h->esz());
        if (rc) return rc;
      }
  // Warm up (and tune) every model at each of its candidate sizes before the clock starts.
  for (int m : sel) {
    const rafiki_greedy_policy& p = policies[m];
    for (int i = 0; i < p.n_sizes; ++i) {
      const int b = p.batch_sizes[i];
      if (b > n) break;
      Model& M = h->models[m];
      rc = stage(h, requests, b, M.stream, M.d_staged_own);
      if (!rc) rc = tune(h, b, model_input(h, requests, M.d_staged_own), M.stream);
      if (!rc) rc = launch_single(h, m, requests, b, out_probs, out_labels);
      if (rc) return rc;
      HIPCHK(hipStreamSynchronize(M.stream));
    }
  }
  struct Busy { bool on = false; int64_t first = 0, b = 0, disp = -1; };
  std::vector<Busy> busy(h->n_models);
  std::vector<rafiki_dispatch> log;
  int64_t head = 0, arrived = 0;
  const int64_t* a = arrival_us;
  ServeClock clk;
  for (;;) {
    // completions
    bool any_busy = false;
    for (int m : sel) {
      Busy& B = busy[m];
      if (!B.on) continue;
      const hipError_t q = hipEventQuery(h->models[m].done);
      if (q == hipErrorNotReady) {   // still running; clear the status so a later launch check does not see it
        (void)hipGetLastError();
        any_busy = true;
        continue;
      }
      if (q != hipSuccess) return fail(RAFIKI_ERR_HIP, std::string("hipEventQuery: ") + hipGetErrorString(q));
      const int64_t done = clk.now();
      for (int64_t i = B.first; i < B.first + B.b; ++i) out_latency_us[i] = done - a[i];
      log[B.disp].end_us = done;
      B.on = false;
    }
    const int64_t t = clk.now();
    while (arrived < n && a[arrived] <= t) ++arrived;
    // dispatch to free models in index order
    for (int m : sel) {
      if (busy[m].on || arrived == head) continue;
      const rafiki_greedy_policy& p = policies[m];
      const int64_t qlen = arrived - head, wait = t - a[head];
      const int32_t b = greedy_decide(p, qlen, wait);
      if (b == 0) continue;
      rc = launch_single(h, m, request_row(h, requests, head), b, out_probs + (size_t)head * C, out_labels + head);
      if (rc) return rc;
      busy[m] = {true, head, b, (int64_t)log.size()};
      log.push_back({t, -1, head, qlen, wait, b, m});
      any_busy = true;
      head += b;
    }
    if (head == n && !any_busy) break;
    // next instant at which a decision can change
    int64_t next = arrived < n ? a[arrived] : INT64_MAX;
    if (arrived > head)
      for (int m : sel)
        if (!busy[m].on) next = std::min(next, greedy_deadline(policies[m], arrived - head, a[head]));
    if (any_busy) next = std::min(next, clk.now() + 20);   // poll running batches
    if (next == INT64_MAX) break;   // nothing running, nothing servable, nothing arriving
    clk.wait_until(next);
  }
  for (size_t i = 0; i < log.size(); ++i) {
    if (i < (size_t)dispatch_cap) out_dispatch[i] = log[i];
  }
  *out_n_dispatch = (int64_t)log.size();
  return RAFIKI_OK;
}

}  // extern "C"
