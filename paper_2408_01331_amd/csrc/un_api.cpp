// Host side of the fused N-model training step: spec validation, the planner
// (fused blocks, depth-level schedule, one device arena, device descriptor
// tables), the step executor and the C ABI declared in unifiednn.h.
//
// Plan overview (UnifiedNN, Model Unifier, Algorithm 1: the hybrid is the
// disjoint union of the sub-models' graphs with one global input):
//   * every parameterised layer plus the ReLU / MaxPool that follow it becomes
//     one fused block; block j of every model forms depth level j;
//   * a step (Trainer, Algorithm 2) is: forward levels 0..L-1, one softmax-CE
//     launch for all models, backward levels L-1..0 (dgrad and wgrad of one
//     level share a launch), one multi-tensor SGD launch;
//   * the first hidden Linear layers of all models read the same input, so
//     their weights live in one concatenated matrix and run as ONE GEMM.
#include "../../include/unifiednn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

// Multi-tile halo forward workgroups: at most UN_HALO_MT m-tiles each, as
// many as leave about UN_HALO_WPS workgroups per slot (two per CU).
#ifndef UN_HALO_MT
#define UN_HALO_MT 4
#endif
#ifndef UN_HALO_WPS
#define UN_HALO_WPS 4
#endif

using namespace un;

namespace {

constexpr size_t NONE = ~(size_t)0;

inline int64_t rup(int64_t x, int64_t a) { return (x + a - 1) / a * a; }
inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

struct Block {
  int kind = 0;  // 0 linear, 1 conv, 2 self-attention core (between its two projections)
  int tokens = 1;  // a Linear on a sequence acts on every token: its GEMM rows are batch * tokens
  int level = 0, model = 0;
  bool relu = false, pool = false, last = false, prev_relu = false, concat = false;
  bool next_linear = false;  // the following block is a Linear (needs transposed output)
  // residual blocks: on the block that ends one, the index of the block whose
  // input is added to its output (res_from); on that first block, the index
  // of the end block, whose output gradient joins its input gradient (res_to)
  int res_from = -1, res_to = -1;
  // linear
  int K = 0, N = 0;
  int in_c = 0, in_h = 1, in_w = 1;  // input viewed as an image (Flatten order mapping)
  // conv
  int C = 0, H = 0, W = 0, O = 0, KH = 0, pad = 0, OH = 0, OW = 0, PH = 0, PW = 0;
  int Cr = 0;  // the model's input channels; C (stored channels) is larger for a padded network input
  // PyTorch-layout offsets in the model's flat parameter vector
  size_t pt_w = 0, pt_b = 0, n_w = 0, n_b = 0;
  // arena offsets (NONE = absent)
  size_t W32 = NONE, b32 = NONE, gW = NONE, gb = NONE, Wb = NONE;
  size_t WT = NONE;        // conv: transposed weights [c][(tap, o)] of the data gradient
  // optimizer state, offsets in the context's state allocation (same layouts as W32 / b32)
  size_t S1 = NONE, S1b = NONE, S2 = NONE, S2b = NONE;
  int64_t ldw = 0, ldwt = 0;
  int rows = 0;            // logical weight rows (N or O)
  size_t X = NONE;         // input (the previous block's output), row-major
  int64_t ldx = 0;
  size_t Y = NONE, amax = NONE;
  size_t P = NONE;         // attention core: softmax probabilities [batch][T][T] fp32
  int64_t ldy = 0;
  size_t G = NONE;         // gradient at this block's output, row-major
  int64_t ldg = 0;
  size_t ws = NONE, ws_size = 0;
  int64_t ldws = 0;
  int splits = 1, kchunk = 0;
  // split-K of a long logits product (forward): its partials, summed by the
  // softmax-CE row pass
  size_t fws = NONE, fws_size = 0;
  int64_t fldws = 0;
  int fsplits = 0, fkchunk = 0;
  // output geometry
  int out_elems_per_sample() const { return kind == 0 ? N : (pool ? PH * PW * O : OH * OW * O); }
};

struct Model {
  std::vector<Block> blocks;
  int num_classes = 0;
  size_t n_params = 0;
  uint64_t seed = 0;
  int group = 0;         // its input group
  int64_t lab_own = 0;   // its own label row (per-model labels): ydev + lab_own int32 elements
};

// One input group: a dataset with its own batch and sample shape, copied to
// the device once per batch and read by every model of the group (Memory
// conservation: a common dataset is loaded only once). One group is the
// shared-input case; a group per model gives every model its own data.
struct Group {
  int B = 0, in_c = 0, in_h = 0, in_w = 0;
  int64_t in_feat = 0, ldxin = 0;
  int in_cs = 0;                    // stored channels of XinC
  size_t xstage = NONE, Xin = NONE, XinC = NONE;
  int64_t lab_shared = 0;           // its label row: ydev + lab_shared int32 elements
  int min_classes = 1 << 30;        // of its models (labels are checked against it)
  bool loaded = false;
  // the first hidden Linear layers of its models read the same input: their
  // weights form one concatenated matrix, one GEMM problem per run of active models
  int64_t kin_p = 0, cat_rows = 0;
  std::vector<int> cat;             // models in the concatenation
  size_t catW32 = NONE, catb32 = NONE, catgW = NONE, catgb = NONE, catWb = NONE, catY = NONE, catG = NONE;
  size_t cat_row_model = NONE;      // int32 per concatenated row: the model owning it
  size_t catS1 = NONE, catS1b = NONE, catS2 = NONE, catS2b = NONE;  // optimizer state (sbase)
};

struct Launch {
  int kind;   // 0 gemm, 1 conv fwd, 2 conv dgrad, 3 conv wgrad, 4 reduce, 5 ce, 6 sgd, 7/8 halo conv fwd/dgrad
  int kclass;
  size_t probs, map;  // arena offsets
  int count;
  int mode = 0;       // conv weight gradient: code variant (launch_conv_wgrad); CE: problems needing the row pass
  size_t lds = 0;     // halo conv: dynamic LDS bytes
};

struct EventRec {
  int kclass;
  hipEvent_t a, b;
};

thread_local std::string g_create_error;

constexpr size_t UN_SCRATCH_BYTES = (size_t)32 << 20;
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[MAX_DEVICES] = {};

}  // namespace

// Workspace of un_step_scratch, one array per device for the life of the
// process. In host code `scratch` is only a stand-in for the device array:
// its device address comes from hipGetSymbolAddress (scratch_on), once per
// device, and only that address is ever handed to kernels.
static __device__ __align__(256) char scratch[UN_SCRATCH_BYTES];

struct un_ctx {
  bool bf16 = false;
  std::vector<Group> groups;
  int maxB = 0;                      // largest batch over the groups
  int64_t lab_elems = 0;             // int32 labels: one row per group, then one per model
  std::vector<Model> models;
  int levels = 0;
  // arena
  char* base = nullptr;
  size_t bytes = 0;
  hipStream_t stream = nullptr;      // the stream every call runs on
  hipStream_t own_stream = nullptr;  // created with the context (stream differs after un_set_stream)
  int device = 0;
  // workspace: the buffers a step writes and reads back within the step only
  // (conv split-K partials, loss partials), one contiguous arena range;
  // wsoff relocates them (un_step_scratch), 0 otherwise
  size_t ws_lo = 0, ws_bytes = 0;
  int64_t wsoff = 0;
  // a captured step (un_graph_capture)
  hipGraph_t graph = nullptr;
  hipGraphExec_t gexec = nullptr;
  bool graph_valid = false;
  bool graph_keep = false, graph_labels = false;  // keep_grads / per-model labels when captured
  // fixed buffers
  size_t ydev = NONE, losses_dev = NONE, ce_partial = NONE;
  size_t lr_dev = NONE;          // per-model learning rates of the current un_step_lr call
  const float* lrv = nullptr;    // lr_dev while such a step is being launched, else null (one rate)
  bool labels_per_model = false; // models read their own label rows (un_load_labels), not their group's
  // optimizers (un_set_optimizer): kind and hyper-parameters per model, and
  // the number of updates each model has taken under it
  struct Opt {
    int kind = UN_OPT_SGD;
    double momentum = 0, beta1 = 0.9, beta2 = 0.999, eps = 1e-8;
    int64_t t = 0;
  };
  std::vector<Opt> opts;
  bool any_opt = false;          // some model is not plain SGD: the step uploads OptHp per model
  char* sbase = nullptr;         // optimizer state (allocated when first needed)
  size_t sbytes = 0;
  size_t opt_dev = NONE;         // OptHp per model
  const OptHp* optp = nullptr;   // opt_dev while a step with optimizers is being launched
  // schedule
  std::vector<Launch> fwd, bwd;
  Launch ce{}, refresh{};
  std::vector<std::pair<int, int>> refresh_rng;  // per model: its tiles [first, first + count) of `refresh`
  std::vector<char> active;          // models in the step (un_set_active)
  size_t tables_off = NONE, tables_cap = 0;  // arena region of the descriptor tables
  std::vector<int64_t> cat_off;      // per model: its first row in its group's concatenation (-1: not in it)
  bool keep_grads = false, grads_valid = false;
  int ce_count = 0;
  bool stepped = false, poisoned = false;
  bool all_loaded() const {
    for (auto& g : groups)
      if (!g.loaded) return false;
    return true;
  }
  std::string err;
  // profiling
  bool profiling = false;
  std::vector<EventRec> recs;
  std::vector<hipEvent_t> free_events;
  double prof_ms[UN_K_COUNT] = {0};
  int64_t prof_n[UN_K_COUNT] = {0};

  template <class T> T* at(size_t off) const { return off == NONE ? nullptr : (T*)(base + off); }
};

namespace {

un_status fail(un_ctx* c, un_status s, const std::string& msg) {
  if (c) c->err = msg;
  else g_create_error = msg;
  return s;
}

#define HIPCHK(ctx, expr)                                                                   \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) {                                                                 \
      (ctx)->poisoned = true;                                                               \
      return fail((ctx), UN_ERR_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    }                                                                                       \
  } while (0)

// --------------------------------------------------------------------------
// Spec parsing
// --------------------------------------------------------------------------
un_status parse_model(const un_model_spec& s, const un_input_spec& in, int mi, Model& m, std::string& why) {
  if (s.n_layers <= 0 || !s.layers) {
    why = "model " + std::to_string(mi) + ": no layers";
    return UN_ERR_INVALID;
  }
  if (s.num_classes <= 0) {
    why = "model " + std::to_string(mi) + ": num_classes must be positive";
    return UN_ERR_INVALID;
  }
  m.num_classes = s.num_classes;
  m.seed = s.init_seed;
  // current shape: image (c, h, w) or flat (f); flat keeps the image it came from
  // The input is an image [c, h, w]; a Linear may read it directly only when
  // h = w = 1. After a Flatten or a Linear the tensor is flat.
  int c = in.in_c, h = in.in_h, w = in.in_w;
  bool flat = false;
  int seq = 0;            // a sequence of `seq` tokens of c features (h = w = 1)
  bool torch_order = in.in_h == 1 && in.in_w == 1;  // flat storage equals PyTorch's flatten order
  size_t pt = 0;
  int i = 0;
  int res_open = -1, res_c = 0, res_h = 0, res_w = 0;  // first block and input shape of an open residual block
  auto where = [&](int li) { return "model " + std::to_string(mi) + " layer " + std::to_string(li) + ": "; };
  while (i < s.n_layers) {
    const un_layer& L = s.layers[i];
    if (L.op == UN_RESIDUAL_BEGIN) {
      if (res_open >= 0) {
        why = where(i) + "nested residual blocks are not supported";
        return UN_ERR_UNSUPPORTED;
      }
      // the skip reads the first enclosed block's input: a block's output, or
      // the network's input when that is flat or a sequence (an image input
      // is staged channel-padded for the convolutions)
      if ((m.blocks.empty() && !(seq || (h == 1 && w == 1))) || s.layers[i - 1].op == UN_FLATTEN) {
        why = where(i) + "a residual block must start at the output of a Linear, Conv2d or attention block, "
                         "or at a flat or sequence input";
        return UN_ERR_UNSUPPORTED;
      }
      res_open = (int)m.blocks.size();
      res_c = c;
      res_h = h;
      res_w = w;
      ++i;
      continue;
    }
    if (L.op == UN_RESIDUAL_END) {
      if (res_open < 0) {
        why = where(i) + "residual end without a begin";
        return UN_ERR_INVALID;
      }
      if ((int)m.blocks.size() == res_open) {
        why = where(i) + "empty residual block";
        return UN_ERR_INVALID;
      }
      if (s.layers[i - 1].op != UN_LINEAR && s.layers[i - 1].op != UN_CONV2D && s.layers[i - 1].op != UN_SELF_ATTENTION) {
        why = where(i) + "a residual block must end with a Linear, Conv2d or attention (a ReLU goes after the end marker)";
        return UN_ERR_UNSUPPORTED;
      }
      Block& e = m.blocks.back();
      if (e.kind == 0 ? (e.N != res_c || e.tokens != std::max(seq, 1)) : (e.O != res_c || e.OH != res_h || e.OW != res_w)) {
        why = where(i) + "a residual block's output shape differs from its input's";
        return UN_ERR_INVALID;
      }
      e.res_from = res_open;
      m.blocks[res_open].res_to = (int)m.blocks.size() - 1;
      res_open = -1;
      ++i;
      if (i < s.n_layers && s.layers[i].op == UN_RELU) {
        e.relu = true;
        ++i;
      }
      if (i < s.n_layers && s.layers[i].op == UN_MAXPOOL2) {
        why = where(i) + "max-pool of a residual sum is not supported";
        return UN_ERR_UNSUPPORTED;
      }
      continue;
    }
    if (res_open >= 0 && L.op != UN_LINEAR && L.op != UN_CONV2D && L.op != UN_RELU && L.op != UN_SELF_ATTENTION) {
      why = where(i) + "a residual block may enclose only Linear, Conv2d, attention and ReLU layers";
      return UN_ERR_UNSUPPORTED;
    }
    if (res_open >= 0 && L.op == UN_CONV2D && i + 1 < s.n_layers &&
        (s.layers[i + 1].op == UN_MAXPOOL2 ||
         (s.layers[i + 1].op == UN_RELU && i + 2 < s.n_layers && s.layers[i + 2].op == UN_MAXPOOL2))) {
      why = where(i) + "a residual block may not enclose a max-pool";
      return UN_ERR_UNSUPPORTED;
    }
    if (L.op == UN_CONV2D) {
      if (flat || seq) {
        why = where(i) + "conv needs an image input (got a flat tensor or a sequence)";
        return UN_ERR_INVALID;
      }
      if (L.out <= 0 || L.kernel <= 0 || L.pad < 0) {
        why = where(i) + "bad conv parameters";
        return UN_ERR_INVALID;
      }
      Block b;
      b.kind = 1;
      b.C = c;
      b.Cr = c;
      b.H = h;
      b.W = w;
      b.O = L.out;
      b.KH = L.kernel;
      b.pad = L.pad;
      b.OH = h + 2 * L.pad - L.kernel + 1;
      b.OW = w + 2 * L.pad - L.kernel + 1;
      if (b.OH <= 0 || b.OW <= 0) {
        why = where(i) + "kernel larger than padded input";
        return UN_ERR_INVALID;
      }
      {
        // the conv kernels address each activation, gradient and weight tensor
        // with 32-bit offsets (buffer loads take byte offsets below 2^31), and
        // an output row of elements with 24-bit multiplies
        const int64_t es = in.precision == UN_BF16_F32MASTER ? 2 : 4, lim = (int64_t)1 << 31;
        const int64_t biggest = std::max({(int64_t)in.batch * c * h * w, (int64_t)in.batch * b.O * b.OH * b.OW,
                                          (int64_t)b.O * (L.kernel * L.kernel * c + 8)});
        if (biggest * es >= lim || (int64_t)b.OW * b.O >= ((int64_t)1 << 24) || (int64_t)w * c >= ((int64_t)1 << 24)) {
          why = where(i) + "conv tensors of 2^31 bytes or more, or output rows of 2^24 elements or more, are not supported";
          return UN_ERR_UNSUPPORTED;
        }
      }
      b.n_w = (size_t)b.O * c * L.kernel * L.kernel;
      b.n_b = b.O;
      b.pt_w = pt;
      b.pt_b = pt + b.n_w;
      pt += b.n_w + b.n_b;
      ++i;
      if (i < s.n_layers && s.layers[i].op == UN_RELU) {
        b.relu = true;
        ++i;
      }
      if (i < s.n_layers && s.layers[i].op == UN_MAXPOOL2) {
        b.pool = true;
        b.PH = b.OH / 2;
        b.PW = b.OW / 2;
        if (b.PH <= 0 || b.PW <= 0) {
          why = where(i) + "max-pool of a map smaller than 2x2";
          return UN_ERR_INVALID;
        }
        ++i;
      }
      c = b.O;
      h = b.pool ? b.PH : b.OH;
      w = b.pool ? b.PW : b.OW;
      flat = false;
      m.blocks.push_back(b);
    } else if (L.op == UN_UNFLATTEN) {
      if (seq || !(flat || (h == 1 && w == 1)) || !torch_order) {
        why = where(i) + "unflatten reads the network's flat input or a Linear layer's flat output";
        return UN_ERR_UNSUPPORTED;
      }
      const int F = c * h * w;
      if (L.out <= 0 || F % L.out != 0) {
        why = where(i) + "unflatten: the tokens must divide the features";
        return UN_ERR_INVALID;
      }
      seq = L.out;
      c = F / L.out;
      h = w = 1;
      flat = false;
      if (c % 8 != 0) {
        why = where(i) + "token features must be a multiple of 8";
        return UN_ERR_UNSUPPORTED;
      }
      ++i;
    } else if (L.op == UN_SELF_ATTENTION) {
      if (!seq) {
        why = where(i) + "attention needs a sequence (add an unflatten)";
        return UN_ERR_INVALID;
      }
      const int d = c;
      const size_t lds = attn_lds_bytes(seq, d, true, 4);  // the fp32 layout, the larger one
      if (seq > 64 || lds > (size_t)160 * 1024) {
        why = where(i) + "attention supports up to 64 tokens whose working set fits 160 KiB of LDS";
        return UN_ERR_UNSUPPORTED;
      }
      // in-projection, core, out-projection: three blocks (levels)
      Block bi;
      bi.kind = 0;
      bi.tokens = seq;
      bi.in_c = d;
      bi.K = d;
      bi.N = 3 * d;
      bi.n_w = (size_t)3 * d * d;
      bi.n_b = (size_t)3 * d;
      bi.pt_w = pt;
      bi.pt_b = pt + bi.n_w;
      pt += bi.n_w + bi.n_b;
      m.blocks.push_back(bi);
      Block bc;
      bc.kind = 2;
      bc.tokens = seq;
      bc.K = d;
      bc.N = d;
      m.blocks.push_back(bc);
      Block bo;
      bo.kind = 0;
      bo.tokens = seq;
      bo.in_c = d;
      bo.K = d;
      bo.N = d;
      bo.n_w = (size_t)d * d;
      bo.n_b = (size_t)d;
      bo.pt_w = pt;
      bo.pt_b = pt + bo.n_w;
      pt += bo.n_w + bo.n_b;
      ++i;
      if (i < s.n_layers && s.layers[i].op == UN_RELU) {
        bo.relu = true;
        ++i;
      }
      m.blocks.push_back(bo);
    } else if (L.op == UN_LINEAR) {
      if (!seq && !flat && !(h == 1 && w == 1)) {
        why = where(i) + "linear on an image needs a flatten first";
        return UN_ERR_INVALID;
      }
      if (L.out <= 0) {
        why = where(i) + "bad linear out";
        return UN_ERR_INVALID;
      }
      if (seq && L.out % 8 != 0) {
        why = where(i) + "token features must be a multiple of 8";
        return UN_ERR_UNSUPPORTED;
      }
      Block b;
      b.kind = 0;
      b.tokens = std::max(seq, 1);
      b.in_c = c;
      b.in_h = h;
      b.in_w = w;
      b.K = c * h * w;
      b.N = L.out;
      b.n_w = (size_t)b.N * b.K;
      b.n_b = b.N;
      b.pt_w = pt;
      b.pt_b = pt + b.n_w;
      pt += b.n_w + b.n_b;
      ++i;
      if (i < s.n_layers && s.layers[i].op == UN_RELU) {
        b.relu = true;
        ++i;
      }
      c = b.N;
      h = w = 1;
      flat = !seq;
      torch_order = true;
      m.blocks.push_back(b);
    } else if (L.op == UN_FLATTEN) {
      if (seq) {
        // token by token: the storage [T][d] is already PyTorch's flatten order
        c = seq * c;
        seq = 0;
      } else {
        torch_order = h == 1 && w == 1;
      }
      flat = true;  // keep (c, h, w): the next Linear maps NCHW order onto NHWC storage
      ++i;
    } else if (L.op == UN_RELU || L.op == UN_MAXPOOL2) {
      why = where(i) + "ReLU/MaxPool2 must directly follow a Conv2d/Linear (ReLU) or Conv2d[+ReLU] (pool)";
      return UN_ERR_UNSUPPORTED;
    } else {
      why = where(i) + "unknown op " + std::to_string(L.op);
      return UN_ERR_INVALID;
    }
  }
  if (res_open >= 0) {
    why = "model " + std::to_string(mi) + ": residual block without an end";
    return UN_ERR_INVALID;
  }
  if (m.blocks.empty() || m.blocks.back().kind != 0 || m.blocks.back().tokens != 1) {
    why = "model " + std::to_string(mi) + ": the last layer must be a Linear on flat features";
    return UN_ERR_UNSUPPORTED;
  }
  if (m.blocks.back().res_from >= 0) {
    why = "model " + std::to_string(mi) + ": a residual block may not end at the logits layer";
    return UN_ERR_UNSUPPORTED;
  }
  Block& last = m.blocks.back();
  if (last.relu) {
    why = "model " + std::to_string(mi) + ": ReLU on the logits is not supported";
    return UN_ERR_UNSUPPORTED;
  }
  if (last.N != s.num_classes) {
    why = "model " + std::to_string(mi) + ": last Linear out != num_classes";
    return UN_ERR_INVALID;
  }
  last.last = true;
  for (size_t j = 0; j < m.blocks.size(); ++j) {
    Block& b = m.blocks[j];
    b.level = (int)j;
    b.model = mi;
    b.prev_relu = j > 0 && m.blocks[j - 1].relu;
    b.next_linear = j + 1 < m.blocks.size() && m.blocks[j + 1].kind == 0;
    if (j + 1 < m.blocks.size() && m.blocks[j + 1].kind == 1 && b.kind != 1) {
      why = "model " + std::to_string(mi) + ": Conv2d after Linear is not supported";
      return UN_ERR_UNSUPPORTED;
    }
    if (b.kind == 1 && b.next_linear && (b.out_elems_per_sample() % 8) != 0) {
      why = "model " + std::to_string(mi) + ": flattened conv output must be a multiple of 8 features";
      return UN_ERR_UNSUPPORTED;
    }
  }
  m.n_params = pt;
  return UN_OK;
}

// --------------------------------------------------------------------------
// Arena
// --------------------------------------------------------------------------
struct Arena {
  size_t top = 0;
  size_t take(size_t bytes) {
    size_t off = rup((int64_t)top, 256);
    top = off + rup((int64_t)std::max<size_t>(bytes, 1), 256);
    return off;
  }
};

// splitmix64: counter-based generator of the library's own initialisation.
inline uint64_t splitmix(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

}  // namespace

// ==========================================================================
// XCD-aware dispatch order
// ==========================================================================
// Workgroup b of a launch runs on XCD b % 8 (round-robin dispatch), and each
// XCD starts its workgroups in increasing b. The tiles of a launch are cut
// into groups that share operands (a run of one problem's tiles); groups are
// given out longest first, each to the XCD with the least work so far, and
// the per-XCD lists are interleaved back into launch order, so a group's tiles
// run on one XCD, close together in time, out of that XCD's L2. Short lists
// are padded with empty entries (the workgroup exits at once). The order
// decides where and when a tile runs, never what it computes.
struct TileGroup {
  int32_t prob, first, count;  // tiles [first, first + count) of problem prob
  double cost;                 // estimated time of the whole group
};

static std::vector<int32_t> xcd_order(std::vector<TileGroup> groups) {
  constexpr int NX = 8;
  std::stable_sort(groups.begin(), groups.end(), [](const TileGroup& a, const TileGroup& b) { return a.cost > b.cost; });
  std::vector<std::vector<int32_t>> q(NX);  // (prob, local) pairs per XCD
  double load[NX] = {0};
  for (const TileGroup& g : groups) {
    int x = 0;
    for (int i = 1; i < NX; ++i)
      if (load[i] < load[x]) x = i;
    load[x] += g.cost;
    for (int t = 0; t < g.count; ++t) {
      q[x].push_back(g.prob);
      q[x].push_back(g.first + t);
    }
  }
  size_t len = 0;
  for (auto& v : q) len = std::max(len, v.size() / 2);
  std::vector<int32_t> map(2 * NX * len, -1);
  for (int x = 0; x < NX; ++x)
    for (size_t i = 0; i < q[x].size() / 2; ++i) {
      map[2 * (i * NX + x)] = q[x][2 * i];
      map[2 * (i * NX + x) + 1] = q[x][2 * i + 1];
    }
  return map;
}

// Halo tiling of a conv forward / data-gradient pass (see ConvProb): a tile
// of BM rows must be whole rows of one image or whole images of the pass's
// pixel space, a pooled forward tile must hold whole windows with nothing
// dropped by floor pooling, the operand channels must be whole 16-byte
// vectors, and the staged rows must fit the LDS budget. Otherwise halo = 0
// and the pass gathers its operand per k-block.
static bool try_halo(ConvProb& p, bool bf, bool dgrad, int BM, int BN) {
  const int BK = bf ? CONV_BK_BF16 : CONV_BK_F32, VEC = bf ? 8 : 4;
  const int SH = dgrad ? p.H : p.OH, SW = dgrad ? p.W : p.OW, Cin = dgrad ? p.O : p.C;
  if (Cin % VEC != 0) return false;
  int tr, imgs;
  if (SH * SW >= BM) {
    if (BM % SW != 0) return false;
    tr = BM / SW;
    if (SH % tr != 0) return false;
    imgs = 1;
  } else {
    if (BM % (SH * SW) != 0) return false;
    tr = SH;
    imgs = BM / (SH * SW);
  }
  if (!dgrad && p.pool && (tr % 2 != 0 || SW % 2 != 0 || SH % 2 != 0)) return false;
  const int cb = std::min(Cin, BK);
  const int cs = cb + ((cb / VEC) % 2 == 0 ? VEC : 0);  // odd number of 16-byte chunks per position
  const int hr = tr + p.KH - 1, hc = SW + p.KH - 1;
  if ((int64_t)imgs * hr * hc * cs > halo_elems(bf ? 2 : 4, BN, BK)) return false;
  if (p.KH * p.KH * (cb / VEC) > HALO_QMAX) return false;
  p.halo = 1;
  p.tr = tr;
  p.imgs = imgs;
  p.hr = hr;
  p.hc = hc;
  p.cb = cb;
  p.cs = cs;
  p.bm = BM;
  p.bn = BN;
  // the tile's divisors (the same definitions as the kernel's) and their
  // reciprocals, rounded once here instead of by every workgroup
  const bool wo = !dgrad && p.pool;  // window-ordered rows
  const int per_row = wo ? SW / 2 : SW, per_img = wo ? (tr / 2) * per_row : tr * SW;
  const int cbw_last = Cin - ((Cin - 1) / cb) * cb;
  auto rc = [](int d) { return 1.0f / (float)d; };
  p.rc_img = rc(per_img);
  p.rc_row = rc(per_row);
  p.rc_kh = rc(p.KH);
  p.rc_cpt = rc(cb / VEC);
  p.rc_cpt_last = rc(cbw_last / VEC);
  p.rc_plane = rc(hr * hc);
  p.rc_hc = rc(hc);
  return true;
}

// A halo forward problem that a multi-tile workgroup can run: one channel
// block, wide or narrow tiles (a tall tile's accumulators leave no registers
// for the rows fetched ahead), staged rows within the fetch-ahead registers.
static bool halo_multi_ok(const ConvProb& p, bool bf) {
  const int BM = bf ? CONV_BM_BF16 : CONV_BM_F32, vec = bf ? 8 : 4, nt = bf ? HALO_NT_BF16 : HALO_NT_F32;
  return p.halo && p.C <= p.cb && p.bm <= 2 * BM && (int64_t)p.imgs * p.hr * p.hc * (p.cb / vec) <= (int64_t)HALO_PF * nt;
}

static void plan_halo(ConvProb& p, bool bf, bool dgrad) {
  const int BM = bf ? CONV_BM_BF16 : CONV_BM_F32, BN = bf ? CONV_BN_BF16 : CONV_BN_F32;
  p.halo = 0;
  // at most BN/2 output columns: the narrow tile wastes no half of each
  // product; a large bf16 forward pass takes the tall one (4BM rows), which
  // halves the workgroups whose fixed costs dominate a short K (a first conv
  // has K = 9 * 8)
  if (bf && !dgrad && p.N <= BN / 2 && p.M >= 64 * 4 * BM && try_halo(p, bf, dgrad, 4 * BM, BN / 2)) return;
  if (p.N <= BN / 2 && try_halo(p, bf, dgrad, 2 * BM, BN / 2)) return;
  try_halo(p, bf, dgrad, BM, BN);
}

// ==========================================================================
// Descriptor tables of one step (the models in c->active only)
// ==========================================================================
struct Tables {
  std::vector<char> host;    // tables as uploaded (pointers encoded as arena offset + 1)
  std::vector<size_t> fix;   // byte offsets of the encoded pointer fields
  std::vector<Launch> fwd, bwd;
  Launch ce{}, refresh{};
  std::vector<std::pair<int, int>> refresh_rng;
};

static void build_tables(un_ctx* c, Tables& T) {
  const bool bf = c->bf16;
  const int levels = c->levels;
  const size_t es = bf ? 2 : 4;
  auto sub = [](size_t off, int64_t bytes) { return off == NONE ? NONE : off + (size_t)bytes; };
  // per input group: runs of consecutive active models of its concatenated
  // level-0 GEMM, [first row, rows)
  std::vector<std::vector<std::pair<int64_t, int64_t>>> cat_runs(c->groups.size());
  for (size_t gi = 0; gi < c->groups.size(); ++gi) {
    const Group& g = c->groups[gi];
    auto& runs = cat_runs[gi];
    for (size_t k = 0; k < g.cat.size(); ++k) {
      if (!c->active[g.cat[k]]) continue;
      const int64_t r0 = c->cat_off[g.cat[k]];
      const int64_t r1 = k + 1 < g.cat.size() ? c->cat_off[g.cat[k + 1]] : g.cat_rows;
      if (!runs.empty() && runs.back().first + runs.back().second == r0) runs.back().second += r1 - r0;
      else runs.push_back({r0, r1 - r0});
    }
  }
  std::vector<char>& host_tables = T.host;
  std::vector<size_t>& fix = T.fix;  // byte offsets (in host_tables) of pointer fields to relocate
  std::vector<Launch>& fwd = T.fwd;
  std::vector<Launch>& bwd = T.bwd;
  auto put = [&](const void* src, size_t n) -> size_t {
    size_t off = rup((int64_t)host_tables.size(), 256);
    host_tables.resize(off + n);
    memcpy(host_tables.data() + off, src, n);
    return off;
  };
  // Pointers are encoded as (arena offset + 1) and fixed up after the arena exists.
  auto ptr = [&](size_t off) -> void* { return off == NONE ? nullptr : (void*)(uintptr_t)(off + 1); };
  // Optimizer state lives in its own allocation: plain device pointers (not relocated).
  auto sp = [&](size_t off, int64_t add) -> float* {
    return (c->sbase && off != NONE) ? (float*)(c->sbase + off + (size_t)add) : nullptr;
  };

  const int GBM = bf ? GEMM_BM_BF16 : GEMM_BM_F32, GBN = bf ? GEMM_BN_BF16 : GEMM_BN_F32;
  const int CBM = bf ? CONV_BM_BF16 : CONV_BM_F32, CBN = bf ? CONV_BN_BF16 : CONV_BN_F32;
  // softmax-CE is fused into a model's logits GEMM when a tile holds whole
  // rows of logits; the loss partials of model m start at m * ce_pstride
  const int ce_pstride = cdiv(c->maxB, CE_ROWS);
  auto ce_fused = [&](const Block& b) { return b.kind == 0 && b.N <= GBN && b.fsplits == 0; };

  // Problems of one launch are ordered longest-K first (their tiles are the
  // longest-running), so the ragged tail of a level is made of short tiles.
  // Order affects scheduling only: every tile computes the same values.
  auto emit_gemm = [&](std::vector<GemmProb>& ps, std::vector<Launch>& out, int kclass) {
    if (ps.empty()) return;
    // k length of one tile: K, or one split's chunk
    const int BKg = bf ? GEMM_BK_BF16 : GEMM_BK_F32;
    auto klen = [&](const GemmProb& x) { return x.epi == EPI_WPART ? std::min(x.K, x.kchunk * BKg) : x.K; };
    std::stable_sort(ps.begin(), ps.end(), [&](const GemmProb& x, const GemmProb& y) { return klen(x) > klen(y); });
    // Launch order = problem order (longest K first), then swizzled for the
    // XCDs: the tiles are cut into runs of up to 8 that share A and B tiles
    // (4 m-tiles x 2 n-tiles, or short columns side by side), and every 8
    // consecutive runs are interleaved so that run r lands on XCD r % 8 with
    // its members 8 launch slots apart - they run together on one XCD and read
    // their shared tiles from its L2 once - while the order stays
    // longest-first at the grain of 8 runs.
    std::vector<int32_t> nat;  // (problem, tile) pairs in run order, with run ids
    std::vector<int32_t> run_of;
    int runs = 0;
    for (size_t k = 0; k < ps.size(); ++k) {
      GemmProb& p = ps[k];
      const int tm = cdiv(p.M, GBM), tn = cdiv(p.N, GBN);
      p.tiles_n = tn;
      // a split-K problem's splits are tile sets of their own (entry
      // split * tiles + tile); runs stay within one split
      const int nsp = p.epi == EPI_WPART ? p.splits : 1;
      for (int sp = 0; sp < nsp; ++sp) {
        const int base = sp * tm * tn;
        if (p.M >= 4 * p.N && tm >= 16) {
          // A (M x K) is much the larger operand (the weight gradient of a
          // concatenated first layer): a run is one m-tile's row of n-tiles (up
          // to 16, balanced), so each A tile is read by one XCD
          const int nr = cdiv(tn, 16), rl = cdiv(tn, nr);
          for (int row = 0; row < tm; ++row)
            for (int c0 = 0; c0 < tn; c0 += rl) {
              ++runs;
              for (int col = c0; col < std::min(tn, c0 + rl); ++col) {
                nat.push_back((int32_t)k);
                nat.push_back(base + col * tm + row);
                run_of.push_back(runs - 1);
              }
            }
        } else {
          // runs of up to 8 tiles: 4 m-tiles x 2 n-tiles, or a shorter
          // column with its neighbours. An A tile (128 x K) and a B tile
          // (K x 128) are the same size, and a run of r x c tiles reads r + c
          // of them: 4 x 2 reads 6 where a column of 8 reads 9
          const int rl = std::min(tm, 4), cpr = std::max(1, 8 / rl);
          for (int c0 = 0; c0 < tn; c0 += cpr)
            for (int r0 = 0; r0 < tm; r0 += rl) {
              ++runs;
              for (int col = c0; col < std::min(tn, c0 + cpr); ++col)
                for (int row = r0; row < std::min(tm, r0 + rl); ++row) {
                  nat.push_back((int32_t)k);
                  nat.push_back(base + col * tm + row);
                  run_of.push_back(runs - 1);
                }
            }
        }
      }
    }
    std::vector<std::vector<int32_t>> members(runs);
    for (size_t i = 0; i < run_of.size(); ++i) members[run_of[i]].push_back((int32_t)i);
    std::vector<int32_t> map;
    for (int r0 = 0; r0 < runs; r0 += 8) {
      const int nr = std::min(8, runs - r0);
      size_t longest = 0;
      for (int r = r0; r < r0 + nr; ++r) longest = std::max(longest, members[r].size());
      for (size_t i = 0; i < longest; ++i)
        for (int x = 0; x < 8; ++x) {
          const int r = r0 + x;
          if (x < nr && i < members[r].size()) {
            map.push_back(nat[2 * members[r][i]]);
            map.push_back(nat[2 * members[r][i] + 1]);
          } else {
            map.push_back(-1);  // keeps the next run member on the same XCD
            map.push_back(0);
          }
        }
    }
    size_t po = put(ps.data(), ps.size() * sizeof(GemmProb));
    for (size_t k = 0; k < ps.size(); ++k) {
      size_t b0 = po + k * sizeof(GemmProb);
      for (size_t f : {offsetof(GemmProb, A), offsetof(GemmProb, B), offsetof(GemmProb, C), offsetof(GemmProb, bias),
                       offsetof(GemmProb, mask), offsetof(GemmProb, dbias), offsetof(GemmProb, W), offsetof(GemmProb, Wb),
                       offsetof(GemmProb, bmaster), offsetof(GemmProb, row_model), offsetof(GemmProb, ce_part),
                       offsetof(GemmProb, R), offsetof(GemmProb, ws)})
        fix.push_back(b0 + f);
    }
    size_t mo = put(map.data(), map.size() * 4);
    out.push_back(Launch{0, kclass, po, mo, (int)(map.size() / 2)});
  };
  auto emit_conv_one = [&](std::vector<ConvProb>& ps, std::vector<Launch>& out, int kind, int kclass) {
    if (ps.empty()) return;
    std::stable_sort(ps.begin(), ps.end(),
                     [](const ConvProb& x, const ConvProb& y) { return (int64_t)x.K * x.splits > (int64_t)y.K * y.splits; });
    const int BK = bf ? CONV_BK_BF16 : CONV_BK_F32;
    int64_t total = 0;
    for (ConvProb& p : ps) {
      p.tiles_m = cdiv(p.M, p.bm ? p.bm : CBM);  // halo tiles and narrow weight-gradient tiles set bm
      p.tiles_n = cdiv(p.N, p.halo ? p.bn : CBN);
      total += (int64_t)p.tiles_m * p.tiles_n;
    }
    // halo forward passes that a multi-tile workgroup can run: mt consecutive
    // m-tiles per workgroup
    const int mt = kind == 7 ? (int)std::max<int64_t>(1, std::min<int64_t>(UN_HALO_MT, total / (UN_HALO_WPS * 2 * 256))) : 1;
    std::vector<TileGroup> gs;
    for (size_t k = 0; k < ps.size(); ++k) {
      ConvProb& p = ps[k];
      const int per_split = p.tiles_m * p.tiles_n;
      if (kind == 7 && mt > 1 && halo_multi_ok(p, bf)) {
        p.mt = mt;
        for (int g = 0; g < p.tiles_m; g += mt)
          for (int tn = 0; tn < p.tiles_n; ++tn)
            gs.push_back(TileGroup{(int32_t)k, g * p.tiles_n + tn, 1, (cdiv(p.K, BK) + 2.0) * mt});
      } else if (kind == 3) {
        // weight gradient: one group per split (its tiles read the same pixels)
        for (int sp = 0; sp < p.splits; ++sp)
          gs.push_back(TileGroup{(int32_t)k, sp * per_split, per_split, per_split * (p.kchunk + 1.0)});
      } else {
        // forward / data gradient: tiles in order (n-fastest), one tile per group
        for (int t = 0; t < per_split; ++t) gs.push_back(TileGroup{(int32_t)k, t, 1, cdiv(p.K, BK) + 2.0});
      }
    }
    std::vector<int32_t> map;
    if (kind == 3) {
      map = xcd_order(gs);
    } else {
      for (auto& g : gs) {
        map.push_back(g.prob);
        map.push_back(g.first);
      }
    }
    size_t po = put(ps.data(), ps.size() * sizeof(ConvProb));
    for (size_t k = 0; k < ps.size(); ++k) {
      size_t b0 = po + k * sizeof(ConvProb);
      for (size_t f : {offsetof(ConvProb, X), offsetof(ConvProb, Wt), offsetof(ConvProb, bias), offsetof(ConvProb, P),
                       offsetof(ConvProb, amax), offsetof(ConvProb, G), offsetof(ConvProb, gam),
                       offsetof(ConvProb, Gprev), offsetof(ConvProb, ws), offsetof(ConvProb, R)})
        fix.push_back(b0 + f);
    }
    size_t mo = put(map.data(), map.size() * 4);
    out.push_back(Launch{kind, kclass, po, mo, (int)(map.size() / 2)});
  };
  auto emit_conv = [&](std::vector<ConvProb>& all, std::vector<Launch>& out, int kind, int kclass) {
    if (kind == 1 || kind == 2) {  // forward / data gradient: halo-tiled problems get their own launch per tile shape
      std::vector<ConvProb> halo, plain;
      size_t lds = 0;
      for (auto& p : all) {
        (p.halo ? halo : plain).push_back(p);
        if (p.halo) lds = std::max(lds, halo_lds_bytes(p, bf ? 2 : 4, bf ? CONV_BK_BF16 : CONV_BK_F32, kind == 2));
      }
      emit_conv_one(halo, out, kind == 1 ? 7 : 8, kclass);
      if (!halo.empty()) out.back().lds = lds;
      emit_conv_one(plain, out, kind, kclass);
    } else {
      // weight gradient: one launch per code variant (pooled / unpooled with
      // whole-vector channels, anything else)
      const int vec = bf ? 8 : 4;
      std::vector<ConvProb> by[3];
      for (auto& p : all) {
        const bool whole = p.O % vec == 0 && p.C % vec == 0;
        by[!whole ? 0 : p.pool ? 1 : 2].push_back(p);
      }
      for (int m = 0; m < 3; ++m) {
        // bf16 whole-vector blocks that all have few output channels: 64-row tiles
        bool narrow = bf && m != 0 && !by[m].empty();
        for (auto& p : by[m]) narrow = narrow && p.O <= CONV_WG_NARROW_BM;
        if (narrow)
          for (auto& p : by[m]) p.bm = CONV_WG_NARROW_BM;
        const size_t before = out.size();
        emit_conv_one(by[m], out, kind, kclass);
        if (out.size() > before) out.back().mode = m | (narrow ? WG_NARROW_BIT : 0);
      }
    }
  };

  // attention core: one workgroup per (problem, sample)
  auto emit_attn = [&](std::vector<AttnProb>& ps, std::vector<Launch>& out, int kind) {
    if (ps.empty()) return;
    std::vector<int32_t> map;
    for (size_t k = 0; k < ps.size(); ++k)
      for (int b = 0; b < ps[k].B; ++b) {
        map.push_back((int32_t)k);
        map.push_back(b);
      }
    size_t lds = 0;
    for (auto& p : ps) lds = std::max(lds, attn_lds_bytes(p.T, p.d, kind == 10, bf ? 2 : 4));
    size_t po = put(ps.data(), ps.size() * sizeof(AttnProb));
    for (size_t k = 0; k < ps.size(); ++k) {
      size_t b0 = po + k * sizeof(AttnProb);
      for (size_t f : {offsetof(AttnProb, QKV), offsetof(AttnProb, A), offsetof(AttnProb, dA), offsetof(AttnProb, dQKV),
                       offsetof(AttnProb, P)})
        fix.push_back(b0 + f);
    }
    size_t mo = put(map.data(), map.size() * 4);
    out.push_back(Launch{kind, UN_K_ATTN, po, mo, (int)(map.size() / 2)});
    out.back().lds = lds;
  };
  auto conv_base = [&](const Block& b) {
    ConvProb p{};
    p.Nb = c->groups[c->models[b.model].group].B;
    p.C = b.C;
    p.H = b.H;
    p.W = b.W;
    p.O = b.O;
    p.KH = b.KH;
    p.pad = b.pad;
    p.OH = b.OH;
    p.OW = b.OW;
    p.PH = b.PH;
    p.PW = b.PW;
    p.pool = b.pool;
    p.relu = b.relu;
    p.prev_relu = b.prev_relu;
    p.splits = 1;
    p.mt = 1;
    return p;
  };

  // forward levels
  for (int lv = 0; lv < levels; ++lv) {
    std::vector<GemmProb> gp;
    std::vector<ConvProb> cp;
    std::vector<AttnProb> ap;
    std::vector<char> cat_done(c->groups.size(), 0);
    for (auto& m : c->models) {
      if (lv >= (int)m.blocks.size() || !c->active[m.blocks[0].model]) continue;
      const Group& g = c->groups[m.group];
      const int B = g.B;
      Block& b = m.blocks[lv];
      if (b.kind == 0) {
        if (b.concat) {
          // one problem per run of consecutive active models of the group's concatenation
          if (cat_done[m.group]) continue;
          cat_done[m.group] = 1;
          for (const auto& run : cat_runs[m.group]) {
            GemmProb p{};
            p.A = ptr(g.Xin);
            p.lda = g.ldxin;
            p.B = ptr(bf ? sub(g.catWb, run.first * g.kin_p * 2) : sub(g.catW32, run.first * g.kin_p * 4));
            p.ldb = g.kin_p;
            p.M = B;
            p.N = (int)run.second;
            p.K = (int)g.in_feat;
            p.epi = EPI_FWD;
            p.relu = 1;
            p.C = ptr(sub(g.catY, run.first * (int64_t)es));
            p.ldc = g.cat_rows;
            p.bias = (const float*)ptr(sub(g.catb32, run.first * 4));
            gp.push_back(p);
          }
          continue;
        }
        GemmProb p{};
        p.A = ptr(b.X);
        p.lda = b.ldx;
        p.B = ptr(bf ? b.Wb : b.W32);
        p.ldb = b.ldw;
        p.M = B * b.tokens;
        p.N = b.N;
        p.K = b.K;
        p.epi = b.last ? EPI_LOGITS : EPI_FWD;
        p.relu = b.relu;
        p.C = ptr(b.Y);
        p.ldc = b.ldy;
        p.bias = (const float*)ptr(b.b32);
        if (b.res_from >= 0) {
          const Block& rb = m.blocks[b.res_from];
          p.R = ptr(rb.X);
          p.ldr = rb.ldx;
        }
        if (b.last && b.fsplits > 0) {
          // split-K logits: the partial sums of each k-chunk (no bias)
          p.epi = EPI_WPART;
          p.splits = b.fsplits;
          p.kchunk = b.fkchunk;
          p.ws = (float*)ptr(b.fws);
          p.ldws = b.fldws;
        }
        if (b.last && ce_fused(b)) {
          // softmax-CE in the logits GEMM's epilogue: it writes dL/dz
          p.C = ptr(b.G);
          p.ldc = b.ldg;
          p.model = b.model;
          p.ce_part = (float*)ptr(sub(c->ce_partial, (int64_t)b.model * ce_pstride * 4));
          p.lab_shared = (int32_t)g.lab_shared;
          p.lab_own = (int32_t)m.lab_own;
        }
        gp.push_back(p);
      } else if (b.kind == 2) {
        const Block& bi = m.blocks[lv - 1];  // the in-projection: Q | K | V per token row
        AttnProb p{};
        p.QKV = ptr(bi.Y);
        p.ldq = bi.ldy;
        p.A = ptr(b.Y);
        p.lda = b.ldy;
        p.P = (float*)ptr(b.P);
        p.T = b.tokens;
        p.d = b.N;
        p.B = B;
        p.scale = (float)(1.0 / std::sqrt((double)b.N));
        ap.push_back(p);
      } else {
        ConvProb p = conv_base(b);
        p.M = b.pool ? B * b.PH * b.PW * 4 : B * b.OH * b.OW;
        p.N = b.O;
        p.K = b.KH * b.KH * b.C;
        p.X = ptr(b.X);
        p.Wt = ptr(bf ? b.Wb : b.W32);
        p.ldw = b.ldw;
        p.bias = (const float*)ptr(b.b32);
        p.P = ptr(b.Y);
        p.amax = (uint8_t*)ptr(b.amax);
        if (b.res_from >= 0) p.R = ptr(m.blocks[b.res_from].X);
        plan_halo(p, bf, false);
        cp.push_back(p);
      }
    }
    emit_gemm(gp, fwd, UN_K_GEMM_FWD);
    emit_conv(cp, fwd, 1, UN_K_CONV_FWD);
    emit_attn(ap, fwd, 9);
  }

  // softmax-CE: the row pass for the models whose CE is not fused (listed
  // first), the loss sum for all
  std::vector<CeProb> ces;
  int ce_rows = 0;
  for (int pass = 0; pass < 2; ++pass)
    for (size_t mi = 0; mi < c->models.size(); ++mi) {
      if (!c->active[mi]) continue;
      const Model& m = c->models[mi];
      const Group& g = c->groups[m.group];
      const Block& b = m.blocks.back();
      if (ce_fused(b) != (pass == 1)) continue;
      CeProb p{};
      p.logits = (const float*)ptr(b.Y);
      p.ldl = b.ldy;
      p.G = ptr(b.G);
      p.ldg = b.ldg;
      p.C = b.N;
      p.model = (int)mi;
      p.nchunks = pass == 1 ? cdiv(g.B, GBM) : cdiv(g.B, CE_ROWS);
      p.B = g.B;
      p.lab_shared = (int32_t)g.lab_shared;
      p.lab_own = (int32_t)m.lab_own;
      if (b.fsplits > 0) {
        p.parts = (const float*)ptr(b.fws);
        p.ldp = b.fldws;
        p.nparts = b.fsplits;
        p.bias = (const float*)ptr(b.b32);
      }
      ces.push_back(p);
      if (pass == 0) ++ce_rows;
    }
  {
    size_t po = put(ces.data(), ces.size() * sizeof(CeProb));
    for (size_t k = 0; k < ces.size(); ++k) {
      size_t b0 = po + k * sizeof(CeProb);
      for (size_t f : {offsetof(CeProb, logits), offsetof(CeProb, G), offsetof(CeProb, parts), offsetof(CeProb, bias)})
        fix.push_back(b0 + f);
    }
    T.ce = Launch{5, UN_K_CE, po, NONE, (int)ces.size()};
    T.ce.mode = ce_rows;
  }

  // Backward launches, one per level lv from the deepest: the Linear data
  // gradients of level lv and the Linear weight gradients of level lv + 1
  // (at lv == 0 also those of level 0). A block's weights are updated one
  // launch after its data gradient has read them, so no launch both reads and
  // writes the same weights. Conv blocks keep their own per-level launches
  // (data gradient, then split-K weight gradient); the split-K reductions
  // with their updates run in one launch after the last level.
  auto add_wgrad = [&](const Block& b, std::vector<GemmProb>& gp, std::vector<char>& cat_done,
                       std::vector<ReduceProb>& rp) {
    const int gi = c->models[b.model].group;
    const Group& g = c->groups[gi];
    const int B = g.B;
    if (b.concat) {
      // one problem per run of consecutive active models of the group's concatenation
      if (cat_done[gi]) return;
      cat_done[gi] = 1;
      const int64_t kin_p = g.kin_p;
      for (const auto& run : cat_runs[gi]) {
        GemmProb p{};
        p.A = ptr(sub(g.catG, run.first * (int64_t)es));
        p.lda = g.cat_rows;
        p.amode = OP_KMAJ;
        p.B = ptr(g.Xin);
        p.ldb = g.ldxin;
        p.bmode = OP_KMAJ;
        p.M = (int)run.second;
        p.N = (int)g.in_feat + 1;
        p.K = B;
        p.epi = EPI_WGRAD;
        p.nsplit = (int)g.in_feat;
        p.C = ptr(sub(g.catgW, run.first * kin_p * 4));
        p.ldc = kin_p;
        p.dbias = (float*)ptr(sub(g.catgb, run.first * 4));
        p.W = (float*)ptr(sub(g.catW32, run.first * kin_p * 4));
        p.Wb = ptr(sub(g.catWb, run.first * kin_p * 2));
        p.bmaster = (float*)ptr(sub(g.catb32, run.first * 4));
        p.row_model = (const int32_t*)ptr(sub(g.cat_row_model, run.first * 4));
        p.s1 = sp(g.catS1, run.first * kin_p * 4);
        p.s2 = sp(g.catS2, run.first * kin_p * 4);
        p.sb1 = sp(g.catS1b, run.first * 4);
        p.sb2 = sp(g.catS2b, run.first * 4);
        gp.push_back(p);
      }
      return;
    }
    GemmProb p{};
    p.A = ptr(b.G);
    p.lda = b.ldg;
    p.amode = OP_KMAJ;
    p.B = ptr(b.X);
    p.ldb = b.ldx;
    p.bmode = OP_KMAJ;
    p.M = b.N;
    p.N = b.K + 1;
    p.K = B * b.tokens;
    p.epi = EPI_WGRAD;
    p.nsplit = b.K;
    p.C = ptr(b.gW);
    p.ldc = b.ldw;
    p.dbias = (float*)ptr(b.gb);
    p.W = (float*)ptr(b.W32);
    p.Wb = ptr(b.Wb);
    p.bmaster = (float*)ptr(b.b32);
    p.model = b.model;
    p.s1 = sp(b.S1, 0);
    p.s2 = sp(b.S2, 0);
    p.sb1 = sp(b.S1b, 0);
    p.sb2 = sp(b.S2b, 0);
    if (b.splits > 1) {
      // partial sums per k-chunk; the reduction below applies the update
      p.epi = EPI_WPART;
      p.splits = b.splits;
      p.kchunk = b.kchunk;
      p.ws = (float*)ptr(b.ws);
      p.ldws = b.ldws;
      ReduceProb r{};
      r.ws = (const float*)ptr(b.ws);
      r.ldws = b.ldws;
      r.splits = b.splits;
      r.O = b.N;
      r.J = b.K;
      r.C = 1;
      r.gW = (float*)ptr(b.gW);
      r.ldgw = b.ldw;
      r.gb = (float*)ptr(b.gb);
      r.W = (float*)ptr(b.W32);
      r.Wb = ptr(b.Wb);
      r.WT = nullptr;
      r.bmaster = (float*)ptr(b.b32);
      r.model = b.model;
      r.s1 = sp(b.S1, 0);
      r.s2 = sp(b.S2, 0);
      r.sb1 = sp(b.S1b, 0);
      r.sb2 = sp(b.S2b, 0);
      rp.push_back(r);
    }
    gp.push_back(p);
  };
  // the split-K reductions (and their updates) of all levels: one launch at
  // the end of the backward pass. Each block's partials have a workspace
  // range of their own, and no later launch of the step reads the weights of
  // a deeper level (a conv block's data gradient has read them before).
  std::vector<ReduceProb> rp;
  for (int lv = levels - 1; lv >= 0; --lv) {
    std::vector<GemmProb> gp;
    std::vector<ConvProb> dp, wp;
    std::vector<AttnProb> ap;
    std::vector<char> cat_done(c->groups.size(), 0);
    for (auto& m : c->models) {
      if (!c->active[m.blocks[0].model]) continue;
      const int B = c->groups[m.group].B;
      const int depth = (int)m.blocks.size();
      if (lv + 1 < depth && m.blocks[lv + 1].kind == 0) add_wgrad(m.blocks[lv + 1], gp, cat_done, rp);
      if (lv >= depth) continue;
      Block& b = m.blocks[lv];
      if (b.kind == 0) {
        // data gradient (not at level 0): the gradient at the previous block's output
        if (lv > 0) {
          Block& pb = m.blocks[lv - 1];
          GemmProb p{};
          p.A = ptr(b.G);
          p.lda = b.ldg;
          p.B = ptr(bf ? b.Wb : b.W32);
          p.ldb = b.ldw;
          p.bmode = OP_KMAJ;
          p.M = B * b.tokens;
          p.N = b.K;
          p.K = b.N;
          p.epi = EPI_DGRAD;
          p.relu = pb.relu;
          p.mask = ptr(b.X);  // the previous block's stored output, row-major
          p.ldmask = b.ldx;
          p.C = ptr(pb.G);
          p.ldc = pb.kind == 1 ? pb.out_elems_per_sample() : pb.ldg * pb.tokens / b.tokens;
          if (b.res_to >= 0) {
            const Block& eb = m.blocks[b.res_to];
            p.R = ptr(eb.G);
            p.ldr = eb.ldg;
          }
          gp.push_back(p);
        }
        if (lv == 0) add_wgrad(b, gp, cat_done, rp);
      } else if (b.kind == 2) {
        // attention core backward: dA (written by the out-projection's data
        // gradient) -> dQ | dK | dV, the gradient at the in-projection's output
        const Block& bi = m.blocks[lv - 1];
        AttnProb p{};
        p.QKV = ptr(bi.Y);
        p.ldq = bi.ldy;
        p.dA = ptr(b.G);
        p.lda = b.ldg;
        p.dQKV = ptr(bi.G);
        p.P = (float*)ptr(b.P);
        p.T = b.tokens;
        p.d = b.N;
        p.B = B;
        p.scale = (float)(1.0 / std::sqrt((double)b.N));
        ap.push_back(p);
      } else {
        const int J = b.KH * b.KH * b.C;
        if (lv > 0) {
          Block& pb = m.blocks[lv - 1];
          ConvProb p = conv_base(b);
          p.M = B * b.H * b.W;
          p.N = b.C;
          p.K = b.KH * b.KH * b.O;
          p.X = ptr(b.X);
          p.Wt = ptr(b.WT);
          p.ldw = b.ldwt;
          p.G = ptr(b.G);
          p.gam = (const uint8_t*)ptr(b.amax);
          p.Gprev = ptr(pb.G);
          if (b.res_to >= 0) p.R = ptr(m.blocks[b.res_to].G);
          plan_halo(p, bf, true);
          dp.push_back(p);
        }
        ConvProb p = conv_base(b);
        p.M = b.O;
        p.N = J + 1;
        p.K = b.pool ? B * b.PH * b.PW * 4 : B * b.OH * b.OW;
        p.X = ptr(b.X);
        p.G = ptr(b.G);
        p.gam = (const uint8_t*)ptr(b.amax);
        p.ws = (float*)ptr(b.ws);
        p.ldws = b.ldws;
        p.splits = b.splits;
        p.kchunk = b.kchunk;
        wp.push_back(p);
        ReduceProb r{};
        r.ws = (const float*)ptr(b.ws);
        r.ldws = b.ldws;
        r.splits = b.splits;
        r.O = b.O;
        r.J = J;
        r.C = b.C;
        r.gW = (float*)ptr(b.gW);
        r.ldgw = b.ldw;
        r.gb = (float*)ptr(b.gb);
        r.W = (float*)ptr(b.W32);
        r.Wb = ptr(b.Wb);
        r.WT = ptr(b.WT);  // conv: the dgrad launch of this level has completed
        r.ldwt = b.ldwt;
        r.bmaster = (float*)ptr(b.b32);
        r.model = b.model;
        r.s1 = sp(b.S1, 0);
        r.s2 = sp(b.S2, 0);
        r.sb1 = sp(b.S1b, 0);
        r.sb2 = sp(b.S2b, 0);
        rp.push_back(r);
      }
    }
    emit_gemm(gp, bwd, UN_K_GEMM_BWD);
    emit_attn(ap, bwd, 10);
    emit_conv(dp, bwd, 2, UN_K_CONV_DGRAD);
    emit_conv(wp, bwd, 3, UN_K_CONV_WGRAD);
  }
  if (!rp.empty()) {
    std::vector<int32_t> map;
    for (size_t k = 0; k < rp.size(); ++k) {
      rp[k].blk_base = (int32_t)map.size();
      const int nb = cdiv((int64_t)rp[k].O * (rp[k].J + 1), REDUCE_BLOCK);
      for (int t = 0; t < nb; ++t) map.push_back((int32_t)k);
    }
    size_t po = put(rp.data(), rp.size() * sizeof(ReduceProb));
    for (size_t k = 0; k < rp.size(); ++k) {
      size_t b0 = po + k * sizeof(ReduceProb);
      for (size_t f : {offsetof(ReduceProb, ws), offsetof(ReduceProb, gW), offsetof(ReduceProb, gb),
                       offsetof(ReduceProb, W), offsetof(ReduceProb, Wb), offsetof(ReduceProb, WT),
                       offsetof(ReduceProb, bmaster)})
        fix.push_back(b0 + f);
    }
    size_t mo = put(map.data(), map.size() * 4);
    bwd.push_back(Launch{4, UN_K_OTHER, po, mo, (int)map.size()});
  }
  // Copy refresh (after un_set_params / initialisation / a set change):
  // rewrite the bf16 copy (and a conv block's transposed copy) of every weight
  // from the fp32 master.
  {
    std::vector<SgdTensor> ts;
    std::vector<int32_t> map;
    auto add = [&](SgdTensor t) {
      t.tiles_r = cdiv(t.R, SGD_TILE);
      t.tiles_c = cdiv(t.Cc, SGD_TILE);
      t.tile_base = (int32_t)map.size();
      const int nt = t.J * t.tiles_r * t.tiles_c;
      for (int k = 0; k < nt; ++k) map.push_back((int32_t)ts.size());
      ts.push_back(t);
    };
    for (auto& m : c->models) {
      const int first = (int)map.size();
      for (auto& b : m.blocks) {
        SgdTensor w{};
        w.W = (float*)ptr(b.W32);
        w.Wb = ptr(b.Wb);
        if (b.Wb == NONE && b.WT == NONE) continue;  // fp32 Linear: nothing besides the master
        w.WT = ptr(b.WT);
        w.ldw = b.ldw;
        w.ldwt = b.ldwt;
        w.R = b.rows;
        if (b.kind == 0) {
          w.J = 1;
          w.Cc = b.K;
        } else {
          w.J = b.KH * b.KH;
          w.Cc = b.C;
        }
        add(w);
      }
      T.refresh_rng.push_back({first, (int)map.size() - first});
    }
    size_t po = put(ts.data(), ts.size() * sizeof(SgdTensor));
    for (size_t k = 0; k < ts.size(); ++k) {
      size_t b0 = po + k * sizeof(SgdTensor);
      for (size_t f : {offsetof(SgdTensor, W), offsetof(SgdTensor, G), offsetof(SgdTensor, Wb), offsetof(SgdTensor, WT)})
        fix.push_back(b0 + f);
    }
    size_t mo = put(map.data(), map.size() * 4);
    T.refresh = Launch{6, UN_K_SGD, po, mo, (int)map.size()};
  }

}

// Relocate a freshly built table set into the arena's table region, upload it
// (the stream must be idle: the previous tables may still be in use by it
// otherwise) and make it the context's schedule.
static un_status install_tables(un_ctx* c, Tables& T) {
  if (T.host.size() > c->tables_cap)
    return fail(c, UN_ERR_UNSUPPORTED, "schedule tables exceed the reserved region");
  for (size_t f : T.fix) {
    uintptr_t v;
    memcpy(&v, T.host.data() + f, sizeof(v));
    if (v != 0) v = (uintptr_t)(c->base + (v - 1));
    memcpy(T.host.data() + f, &v, sizeof(v));
  }
  auto relocate = [&](Launch& l) {
    l.probs += c->tables_off;
    if (l.map != NONE) l.map += c->tables_off;
  };
  for (auto& l : T.fwd) relocate(l);
  for (auto& l : T.bwd) relocate(l);
  relocate(T.ce);
  relocate(T.refresh);
  HIPCHK(c, hipMemcpyAsync(c->base + c->tables_off, T.host.data(), T.host.size(), hipMemcpyHostToDevice, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  c->fwd = T.fwd;
  c->bwd = T.bwd;
  c->ce = T.ce;
  c->refresh = T.refresh;
  c->refresh_rng = T.refresh_rng;
  c->graph_valid = false;  // a captured step read the previous tables
  return UN_OK;
}

// ==========================================================================
// Planner
// ==========================================================================
// dry: plan only - c->bytes is the arena the context would allocate; nothing
// touches the device.
static un_status plan_and_alloc(un_ctx* c, bool dry = false) {
  const bool bf = c->bf16;
  const size_t es = bf ? 2 : 4;  // storage element size
  Arena A;
  const size_t N = c->models.size();

  // labels: one row per input group (un_load_batch), then one per model (un_load_labels)
  c->lab_elems = 0;
  for (auto& g : c->groups) {
    g.lab_shared = c->lab_elems;
    c->lab_elems += g.B;
  }
  for (auto& m : c->models) {
    m.lab_own = c->lab_elems;
    c->lab_elems += c->groups[m.group].B;
  }
  c->ydev = A.take((size_t)c->lab_elems * 4);
  c->lr_dev = A.take(N * 4);
  c->opt_dev = A.take(N * sizeof(OptHp));
  c->losses_dev = A.take(N * 4);
  c->cat_off.assign(N, -1);
  const int vec = bf ? 8 : 4;
  for (size_t gi = 0; gi < c->groups.size(); ++gi) {
    Group& g = c->groups[gi];
    const int B = g.B;
    g.in_feat = (int64_t)g.in_c * g.in_h * g.in_w;
    g.xstage = A.take((size_t)B * g.in_feat * 4);
    bool any_linear0 = false, any_conv0 = false;
    for (auto& m : c->models) {
      if (m.group != (int)gi) continue;
      if (m.blocks[0].kind == 0) any_linear0 = true;
      else any_conv0 = true;
    }
    // A first conv whose input channels are not a whole number of 16-byte
    // vectors (RGB, grey-scale) reads a copy of the input with zero channels
    // appended: its loaders then take whole vectors, and the padded weight
    // columns meet zeros only, so their gradient is exactly 0 and they stay 0.
    g.in_cs = g.in_c;
    if (any_conv0 && g.in_c % vec != 0) {
      g.in_cs = (int)rup(g.in_c, vec);
      g.XinC = A.take((size_t)B * g.in_h * g.in_w * g.in_cs * es);
      for (auto& m : c->models)
        if (m.group == (int)gi && m.blocks[0].kind == 1) m.blocks[0].C = g.in_cs;
    }
    if (g.XinC == NONE || any_linear0) g.Xin = A.take((size_t)B * g.in_feat * es);
    g.ldxin = g.in_feat;
    if (any_linear0 && g.in_feat % 8 != 0)
      return fail(nullptr, UN_ERR_UNSUPPORTED,
                  "input features must be a multiple of 8 when a model starts with Linear (input group " +
                      std::to_string(gi) + ")");

    // level-0 concatenation: the group's hidden Linear + ReLU first layers
    // whose output is read as flat rows (a sequence view needs rows of one
    // token, which the concatenated output's row stride cannot give) and
    // that add no skip of their own (the joint GEMM has no per-model operand)
    g.cat.clear();
    for (size_t i = 0; i < N; ++i) {
      const auto& bl = c->models[i].blocks;
      const Block& b = bl[0];
      if (c->models[i].group == (int)gi && b.kind == 0 && b.tokens == 1 && !b.last && b.relu && b.res_from < 0 &&
          bl[1].tokens == 1)
        g.cat.push_back((int)i);
    }
    g.cat_rows = 0;
    for (int i : g.cat) {
      c->cat_off[i] = g.cat_rows;
      g.cat_rows += rup(c->models[i].blocks[0].N + 1, 8);  // >= 1 spare row
    }
    g.kin_p = rup(g.in_feat, 8);
    if (!g.cat.empty()) {
      g.catW32 = A.take((size_t)g.cat_rows * g.kin_p * 4);
      g.catb32 = A.take((size_t)g.cat_rows * 4);
      g.catgW = A.take((size_t)g.cat_rows * g.kin_p * 4);
      g.catgb = A.take((size_t)g.cat_rows * 4);
      if (bf) g.catWb = A.take((size_t)g.cat_rows * g.kin_p * 2);
      g.catY = A.take((size_t)B * g.cat_rows * es);
      g.catG = A.take((size_t)B * g.cat_rows * es);
      g.cat_row_model = A.take((size_t)g.cat_rows * 4);
    }
  }

  // --- per block buffers
  int levels = 0;
  for (size_t mi = 0; mi < c->models.size(); ++mi) {
    Model& m = c->models[mi];
    const Group& g = c->groups[m.group];
    const int B = g.B;
    levels = std::max(levels, (int)m.blocks.size());
    for (size_t j = 0; j < m.blocks.size(); ++j) {
      Block& b = m.blocks[j];
      const int64_t R = (int64_t)B * b.tokens;  // GEMM rows: samples, or samples x tokens
      if (b.kind == 2) {
        // attention core: A [R][d] and its gradient, P [B][T][T] fp32; no weights
        b.ldy = b.N;
        b.Y = A.take((size_t)R * b.ldy * es);
        b.ldg = b.N;
        b.G = A.take((size_t)R * b.ldg * es);
        b.P = A.take((size_t)B * b.tokens * b.tokens * 4);
      } else if (b.kind == 0) {
        b.rows = b.N;
        b.ldw = rup(b.K, 8);
        if (j == 0 && c->cat_off[mi] >= 0) {
          b.concat = true;
          const size_t roff = (size_t)c->cat_off[mi];
          b.W32 = g.catW32 + roff * b.ldw * 4;
          b.b32 = g.catb32 + roff * 4;
          b.gW = g.catgW + roff * b.ldw * 4;
          b.gb = g.catgb + roff * 4;
          if (bf) b.Wb = g.catWb + roff * b.ldw * 2;
          b.ldy = g.cat_rows;
          b.Y = g.catY + roff * es;
          b.ldg = g.cat_rows;
          b.G = g.catG + roff * es;
        } else {
          b.W32 = A.take((size_t)b.N * b.ldw * 4);
          b.b32 = A.take((size_t)b.N * 4);
          b.gW = A.take((size_t)b.N * b.ldw * 4);
          b.gb = A.take((size_t)b.N * 4);
          if (bf) b.Wb = A.take((size_t)b.N * b.ldw * 2);
          if (b.last) {
            b.ldy = rup(b.N, 8);
            b.Y = A.take((size_t)R * b.ldy * 4);  // fp32 logits
            // split-K of a long logits contraction with few classes: chunks
            // of at most 8 (fp32: 16) k-blocks, whose partials go to the
            // workspace; the softmax-CE row pass adds them in split order,
            // then the bias. A few tiles with a long K would otherwise run
            // alone at the end of their level; the row pass's work grows with
            // classes x splits, so many classes keep the fused CE. Depends
            // only on this block's shape.
            const int BKf = bf ? GEMM_BK_BF16 : GEMM_BK_F32, FKCH = bf ? 8 : 16;
            const int nkbf = cdiv(b.K, BKf);
            if (nkbf > FKCH && b.N <= 32 && b.tokens == 1) {  // rows = samples (the row pass's layout)
              b.fsplits = cdiv(nkbf, FKCH);
              b.fkchunk = cdiv(nkbf, b.fsplits);
              b.fsplits = cdiv(nkbf, b.fkchunk);
              b.fldws = rup(b.N, 4);
              b.fws_size = (size_t)b.fsplits * R * b.fldws * 4;  // placed in the workspace range below
            }
          } else {
            b.ldy = rup(b.N, 8);
            b.Y = A.take((size_t)R * b.ldy * es);
          }
          b.ldg = rup(b.N, 8);
          b.G = A.take((size_t)R * b.ldg * es);
          // split-K weight gradient for a long contraction (rows = samples x
          // tokens): chunks of at most 16 k-blocks, partials in the workspace,
          // summed in split order by the level's reduction launch, which
          // applies the update. Depends only on this block's shape.
          const int BKg = bf ? GEMM_BK_BF16 : GEMM_BK_F32, KCH = bf ? 16 : 32;
          const int nkb = cdiv(R, BKg);
          if (nkb > KCH) {
            b.splits = cdiv(nkb, KCH);
            b.kchunk = cdiv(nkb, b.splits);
            b.splits = cdiv(nkb, b.kchunk);
            b.ldws = rup(b.K + 1, 4);
            b.ws_size = (size_t)b.splits * b.N * b.ldws * 4;  // placed in the workspace range below
          }
        }
      } else {
        const int J = b.KH * b.KH * b.C;
        b.rows = b.O;
        b.ldw = rup(J, 8);
        b.W32 = A.take((size_t)b.O * b.ldw * 4);
        b.b32 = A.take((size_t)b.O * 4);
        b.gW = A.take((size_t)b.O * b.ldw * 4);
        b.gb = A.take((size_t)b.O * 4);
        if (bf) b.Wb = A.take((size_t)b.O * b.ldw * 2);
        if (j > 0) {
          b.ldwt = rup((int64_t)b.KH * b.KH * b.O, 8);
          b.WT = A.take((size_t)b.C * b.ldwt * es);
        }
        const int64_t npix = (int64_t)B * (b.pool ? b.PH * b.PW : b.OH * b.OW);
        b.Y = A.take((size_t)npix * b.O * es);
        b.ldy = b.O;
        if (b.pool) b.amax = A.take((size_t)npix * b.O);
        b.G = A.take((size_t)npix * b.O * es);
        b.ldg = b.O;
        // split-K of the weight gradient: depends only on this block's shape
        const int BK = bf ? CONV_BK_BF16 : CONV_BK_F32;
        const int BMc = bf ? CONV_BM_BF16 : CONV_BM_F32, BNc = bf ? CONV_BN_BF16 : CONV_BN_F32;
        const int64_t kpix = b.pool ? (int64_t)B * b.PH * b.PW * 4 : (int64_t)B * b.OH * b.OW;
        const int nkb = cdiv(kpix, BK);
        const int tiles = cdiv(b.O, BMc) * cdiv(J + 1, BNc);
        // >= 4 k-blocks per split and at most 64 workgroups: 64 is the
        // concurrent capacity of one XCD (32 CUs x 2), so the problems of a
        // launch fill whole rounds instead of leaving a short extra one.
        // Blocks whose channel counts are not whole 16-byte vectors take the
        // element-wise loaders (several times slower per k-block): chunks of
        // 8 k-blocks, up to 512 workgroups. fp32 blocks with small partials
        // (<= 64 KiB per split): chunks of 16 k-blocks, up to 256 workgroups.
        int splits = std::max(1, std::min(nkb / 4, 64 / tiles));
        const int vec = bf ? 8 : 4;
        if (b.O % vec != 0 || b.C % vec != 0) splits = std::max(splits, std::min(nkb / 8, 512 / tiles));
        else if (!bf && (int64_t)b.O * rup(J + 1, 4) * 4 <= 65536) splits = std::max(splits, std::min(nkb / 16, 256 / tiles));
        b.kchunk = cdiv(nkb, splits);
        b.splits = cdiv(nkb, b.kchunk);
        b.ldws = rup(J + 1, 4);
        b.ws_size = (size_t)b.splits * b.O * b.ldws * 4;  // placed in the workspace range below
      }
    }
    // wire inputs
    for (size_t j = 0; j < m.blocks.size(); ++j) {
      Block& b = m.blocks[j];
      // row strides: a token-wise layer reads rows of one token, a flat one
      // rows of one sample (a sequence's storage [T][d] is its flat view)
      if (j == 0) {
        b.X = (b.kind == 1 && g.XinC != NONE) ? g.XinC : g.Xin;
        b.ldx = b.kind == 1 ? g.ldxin : g.ldxin / b.tokens;
      } else {
        Block& p = m.blocks[j - 1];
        b.X = p.Y;
        b.ldx = p.kind == 1 ? p.out_elems_per_sample() : p.ldy * p.tokens / b.tokens;
      }
    }
  }
  c->levels = levels;

  // --- workspace: one contiguous range (relocatable as a whole, un_step_scratch)
  c->ws_lo = (size_t)rup((int64_t)A.top, 256);
  A.top = c->ws_lo;
  c->ce_partial = A.take(c->models.size() * (size_t)cdiv(c->maxB, CE_ROWS) * 4);
  for (auto& m : c->models)
    for (auto& b : m.blocks)
      {
        if (b.ws_size) b.ws = A.take(b.ws_size);
        if (b.fws_size) b.fws = A.take(b.fws_size);
      }
  c->ws_bytes = A.top - c->ws_lo;

  c->active.assign(c->models.size(), 1);
  Tables T;
  build_tables(c, T);

  // --- allocate the arena: buffers + tables (room for the tables of any
  // active subset, which are never larger than twice the full set's)
  c->tables_cap = 2 * T.host.size() + ((size_t)1 << 20);
  c->tables_off = A.take(c->tables_cap);
  c->bytes = A.top;
  if (dry) return UN_OK;
  hipError_t e = hipMalloc((void**)&c->base, c->bytes);
  if (e != hipSuccess) {
    c->base = nullptr;
    return fail(nullptr, UN_ERR_OOM, "hipMalloc of " + std::to_string(c->bytes) + " bytes failed: " + hipGetErrorString(e));
  }
  HIPCHK(c, hipMemsetAsync(c->base, 0, c->bytes, c->stream));
  {
    un_status st = install_tables(c, T);
    if (st != UN_OK) return st;
  }
  for (auto& g : c->groups) {
    if (!g.cat.empty()) {
      std::vector<int32_t> row_model((size_t)g.cat_rows);
      for (size_t k = 0; k < g.cat.size(); ++k) {
        const int64_t r1 = k + 1 < g.cat.size() ? c->cat_off[g.cat[k + 1]] : g.cat_rows;
        for (int64_t r = c->cat_off[g.cat[k]]; r < r1; ++r) row_model[(size_t)r] = g.cat[k];
      }
      HIPCHK(c, hipMemcpyAsync(c->base + g.cat_row_model, row_model.data(), row_model.size() * 4,
                               hipMemcpyHostToDevice, c->stream));
      HIPCHK(c, hipStreamSynchronize(c->stream));  // row_model is freed at the end of this scope
    }
    // the padding channels of XinC are written here only, once
    if (g.XinC != NONE)
      HIPCHK(c, hipMemsetAsync(c->base + g.XinC, 0, (size_t)g.B * g.in_h * g.in_w * g.in_cs * es, c->stream));
  }
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return UN_OK;
}

// ==========================================================================
// Parameter layout mapping (PyTorch state_dict order <-> internal)
// ==========================================================================
// Internal column of PyTorch weight column `col` for a block.
static inline int64_t lin_col(const Block& b, int64_t col) {
  // PyTorch flattens NCHW: col = c*(h*w) + y*w + x; internal NHWC: (y*w + x)*c_count + c
  const int hw = b.in_h * b.in_w;
  const int64_t ch = col / hw, s = col - ch * hw;
  return s * b.in_c + ch;
}

static void to_internal(const Block& b, const float* pt, std::vector<float>& w, std::vector<float>& bias) {
  if (b.kind == 0) {
    w.assign((size_t)b.N * b.ldw, 0.f);
    for (int o = 0; o < b.N; ++o)
      for (int k = 0; k < b.K; ++k) w[(size_t)o * b.ldw + lin_col(b, k)] = pt[b.pt_w + (size_t)o * b.K + k];
    bias.assign(pt + b.pt_b, pt + b.pt_b + b.N);
  } else {
    w.assign((size_t)b.O * b.ldw, 0.f);
    for (int o = 0; o < b.O; ++o)
      for (int ci = 0; ci < b.Cr; ++ci)
        for (int u = 0; u < b.KH; ++u)
          for (int v = 0; v < b.KH; ++v)
            w[(size_t)o * b.ldw + ((size_t)u * b.KH + v) * b.C + ci] =
                pt[b.pt_w + (((size_t)o * b.Cr + ci) * b.KH + u) * b.KH + v];
    bias.assign(pt + b.pt_b, pt + b.pt_b + b.O);
  }
}

static void from_internal(const Block& b, const std::vector<float>& w, const std::vector<float>& bias, float* pt) {
  if (b.kind == 0) {
    for (int o = 0; o < b.N; ++o)
      for (int k = 0; k < b.K; ++k) pt[b.pt_w + (size_t)o * b.K + k] = w[(size_t)o * b.ldw + lin_col(b, k)];
    std::copy(bias.begin(), bias.end(), pt + b.pt_b);
  } else {
    for (int o = 0; o < b.O; ++o)
      for (int ci = 0; ci < b.Cr; ++ci)
        for (int u = 0; u < b.KH; ++u)
          for (int v = 0; v < b.KH; ++v)
            pt[b.pt_w + (((size_t)o * b.Cr + ci) * b.KH + u) * b.KH + v] =
                w[(size_t)o * b.ldw + ((size_t)u * b.KH + v) * b.C + ci];
    std::copy(bias.begin(), bias.end(), pt + b.pt_b);
  }
}

// Rewrite the bf16 (and conv transposed) weight copies from the fp32 master:
// of every model, or of model i only.
static un_status refresh_copies(un_ctx* c, int i = -1) {
  const Launch& l = c->refresh;
  const int blk0 = i < 0 ? 0 : c->refresh_rng[i].first, n = i < 0 ? l.count : c->refresh_rng[i].second;
  HIPCHK(c, launch_sgd(c->bf16, c->at<SgdTensor>(l.probs), c->at<int32_t>(l.map), blk0, n, 0.f, false, c->stream));
  return UN_OK;
}

// Model i's tensors of one kind (weights and biases at the Block offsets wf,
// bf from `base`) from / to the PyTorch layout.
static un_status write_blocks(un_ctx* c, int i, char* base, size_t Block::*wf, size_t Block::*bf, const float* src) {
  Model& m = c->models[i];
  std::vector<float> w, bias;
  for (auto& b : m.blocks) {
    if (b.kind == 2) continue;  // the attention core has no parameters
    to_internal(b, src, w, bias);
    // on the context's stream, completed before the host buffers go away
    HIPCHK(c, hipMemcpyAsync(base + b.*wf, w.data(), w.size() * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipMemcpyAsync(base + b.*bf, bias.data(), bias.size() * 4, hipMemcpyHostToDevice, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
  }
  return UN_OK;
}

static un_status read_blocks(un_ctx* c, int i, const char* base, size_t Block::*wf, size_t Block::*bf, float* dst) {
  Model& m = c->models[i];
  HIPCHK(c, hipStreamSynchronize(c->stream));
  std::vector<float> w, bias;
  for (auto& b : m.blocks) {
    if (b.kind == 2) continue;
    w.resize((size_t)b.rows * b.ldw);
    bias.resize(b.rows);
    HIPCHK(c, hipMemcpyAsync(w.data(), base + b.*wf, w.size() * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipMemcpyAsync(bias.data(), base + b.*bf, bias.size() * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    from_internal(b, w, bias, dst);
  }
  return UN_OK;
}

static un_status write_params(un_ctx* c, int i, const float* src) {
  return write_blocks(c, i, c->base, &Block::W32, &Block::b32, src);
}

static un_status read_tensors(un_ctx* c, int i, bool grads, float* dst) {
  return grads ? read_blocks(c, i, c->base, &Block::gW, &Block::gb, dst)
               : read_blocks(c, i, c->base, &Block::W32, &Block::b32, dst);
}

// Library initialisation: Kaiming-uniform weights, U(+-1/sqrt(fan_in)) biases,
// uniforms from splitmix64(seed, tensor, element).
static void init_host(const Model& m, std::vector<float>& pt) {
  pt.assign(m.n_params, 0.f);
  int t = 0;
  for (auto& b : m.blocks) {
    if (b.kind == 2) continue;
    const double fan_in = b.kind == 0 ? (double)b.K : (double)b.Cr * b.KH * b.KH;
    const double wb = std::sqrt(6.0 / fan_in), bb = 1.0 / std::sqrt(fan_in);
    for (int part = 0; part < 2; ++part, ++t) {
      const size_t off = part == 0 ? b.pt_w : b.pt_b, n = part == 0 ? b.n_w : b.n_b;
      const double bound = part == 0 ? wb : bb;
      for (size_t e = 0; e < n; ++e) {
        const uint64_t r = splitmix(m.seed ^ splitmix(((uint64_t)t << 40) ^ e));
        const double u = (double)(r >> 11) * (1.0 / 9007199254740992.0);  // [0, 1)
        pt[off + e] = (float)((2.0 * u - 1.0) * bound);
      }
    }
  }
}

// ==========================================================================
// Execution
// ==========================================================================
static hipError_t run_launch(un_ctx* c, const Launch& l, float lr) {
  hipEvent_t a = nullptr, b = nullptr;
  if (c->profiling) {
    auto get = [&]() {
      hipEvent_t e = nullptr;
      if (!c->free_events.empty()) {
        e = c->free_events.back();
        c->free_events.pop_back();
      } else if (hipEventCreate(&e) != hipSuccess) {
        e = nullptr;
      }
      return e;
    };
    a = get();
    b = get();
    if (a) hipEventRecord(a, c->stream);
  }
  hipError_t e = hipSuccess;
  switch (l.kind) {
    case 0:
      e = launch_gemm(c->bf16, l.kclass == UN_K_GEMM_BWD, c->at<GemmProb>(l.probs), c->at<int32_t>(l.map), l.count, lr,
                      c->lrv, c->optp, c->keep_grads, c->at<int32_t>(c->ydev), c->labels_per_model, c->wsoff,
                      c->stream);
      break;
    case 1:
      e = launch_conv_fwd(c->bf16, c->at<ConvProb>(l.probs), c->at<int32_t>(l.map), l.count, c->stream);
      break;
    case 2:
      e = launch_conv_dgrad(c->bf16, c->at<ConvProb>(l.probs), c->at<int32_t>(l.map), l.count, c->stream);
      break;
    case 3:
      e = launch_conv_wgrad(c->bf16, l.mode, c->at<ConvProb>(l.probs), c->at<int32_t>(l.map), l.count, c->wsoff,
                            c->stream);
      break;
    case 7:
    case 8:
      e = launch_conv_halo(c->bf16, l.kind == 8, c->at<ConvProb>(l.probs), c->at<int32_t>(l.map), l.count, l.lds,
                           c->stream);
      break;
    case 4:
      e = launch_reduce(c->bf16, c->at<ReduceProb>(l.probs), c->at<int32_t>(l.map), l.count, lr, c->lrv, c->optp,
                        c->keep_grads, c->wsoff, c->stream);
      break;
    case 5:
      e = launch_ce(c->bf16, c->at<CeProb>(l.probs), l.count, l.mode, c->at<int32_t>(c->ydev), c->labels_per_model,
                    c->maxB, (float*)((char*)c->at<float>(c->ce_partial) + c->wsoff), cdiv(c->maxB, CE_ROWS),
                    c->at<float>(c->losses_dev), c->wsoff, c->stream);
      break;
    case 6:
      e = launch_sgd(c->bf16, c->at<SgdTensor>(l.probs), c->at<int32_t>(l.map), 0, l.count, lr, true, c->stream);
      break;
    case 9:
    case 10:
      e = launch_attn(c->bf16, l.kind == 10, c->at<AttnProb>(l.probs), c->at<int32_t>(l.map), l.count, l.lds,
                      c->stream);
      break;
  }
  if (c->profiling && a && b) {
    hipEventRecord(b, c->stream);
    c->recs.push_back(EventRec{l.kclass, a, b});
  }
  return e;
}

static un_status drain_profile(un_ctx* c) {
  if (c->recs.empty()) return UN_OK;
  HIPCHK(c, hipStreamSynchronize(c->stream));
  for (auto& r : c->recs) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      c->prof_ms[r.kclass] += ms;
      c->prof_n[r.kclass] += 1;
    }
    c->free_events.push_back(r.a);
    c->free_events.push_back(r.b);
  }
  c->recs.clear();
  return UN_OK;
}

#define CHECK_CTX(c)                                                         \
  do {                                                                       \
    if (!(c)) return fail(nullptr, UN_ERR_INVALID, "null context");          \
    if ((c)->poisoned) return fail((c), UN_ERR_DEVICE, "context poisoned by an earlier device error"); \
  } while (0)

// ==========================================================================
// C ABI
// ==========================================================================
extern "C" {

static size_t state_layout(un_ctx* c);

// Validation and parsing shared by un_create and un_plan_bytes: a context
// with its models parsed and nothing on the device.
static un_status parse_all(const un_model_spec* specs, int32_t n_models, const un_input_spec* ins, int32_t n_groups,
                           const int32_t* group_of, un_ctx** out) {
  *out = nullptr;
  if (!specs || !ins || n_models <= 0) return fail(nullptr, UN_ERR_INVALID, "specs/inputs NULL or n_models <= 0");
  if (n_groups <= 0 || n_groups > n_models) return fail(nullptr, UN_ERR_INVALID, "need 1 <= n_groups <= n_models");
  if (n_groups > 1 && !group_of) return fail(nullptr, UN_ERR_INVALID, "group_of is NULL with several input groups");
  for (int g = 0; g < n_groups; ++g) {
    const un_input_spec& in = ins[g];
    if (in.batch <= 0 || in.in_c <= 0 || in.in_h <= 0 || in.in_w <= 0)
      return fail(nullptr, UN_ERR_INVALID, "input group " + std::to_string(g) + ": dimensions must be positive");
    if (in.batch > CE_MAX_BATCH) return fail(nullptr, UN_ERR_UNSUPPORTED, "batch larger than 2^20");
    if (in.precision != UN_F32 && in.precision != UN_BF16_F32MASTER)
      return fail(nullptr, UN_ERR_INVALID, "unknown precision");
    if (in.precision != ins[0].precision)
      return fail(nullptr, UN_ERR_INVALID, "every input group must have the same precision");
  }
  std::vector<int> used(n_groups, 0);
  for (int i = 0; i < n_models; ++i) {
    const int g = group_of ? group_of[i] : 0;
    if (g < 0 || g >= n_groups)
      return fail(nullptr, UN_ERR_RANGE, "model " + std::to_string(i) + ": input group out of range");
    used[g] = 1;
  }
  for (int g = 0; g < n_groups; ++g)
    if (!used[g]) return fail(nullptr, UN_ERR_INVALID, "input group " + std::to_string(g) + " has no model");
  un_ctx* c = new un_ctx();
  c->bf16 = ins[0].precision == UN_BF16_F32MASTER;
  c->groups.resize(n_groups);
  for (int g = 0; g < n_groups; ++g) {
    Group& gr = c->groups[g];
    gr.B = ins[g].batch;
    gr.in_c = ins[g].in_c;
    gr.in_h = ins[g].in_h;
    gr.in_w = ins[g].in_w;
    c->maxB = std::max(c->maxB, gr.B);
  }
  c->models.resize(n_models);
  c->opts.resize(n_models);
  for (int i = 0; i < n_models; ++i) {
    const int g = group_of ? group_of[i] : 0;
    std::string why;
    un_status s = parse_model(specs[i], ins[g], i, c->models[i], why);
    if (s != UN_OK) {
      delete c;
      return fail(nullptr, s, why);
    }
    c->models[i].group = g;
    c->groups[g].min_classes = std::min(c->groups[g].min_classes, c->models[i].num_classes);
  }
  *out = c;
  return UN_OK;
}

un_status un_plan_bytes_grouped(const un_model_spec* specs, int32_t n_models, const un_input_spec* inputs,
                                int32_t n_groups, const int32_t* group_of, size_t* arena_bytes, size_t* state_bytes) {
  if (!arena_bytes) return fail(nullptr, UN_ERR_INVALID, "arena_bytes is NULL");
  un_ctx* c = nullptr;
  un_status s = parse_all(specs, n_models, inputs, n_groups, group_of, &c);
  if (s != UN_OK) return s;
  s = plan_and_alloc(c, true);
  if (s == UN_OK) {
    *arena_bytes = c->bytes;
    if (state_bytes) *state_bytes = state_layout(c);
  } else {
    const std::string msg = c->err.empty() ? g_create_error : c->err;
    delete c;
    return fail(nullptr, s, msg);
  }
  delete c;
  return UN_OK;
}

un_status un_plan_bytes(const un_model_spec* specs, int32_t n_models, const un_input_spec* in, size_t* arena_bytes,
                        size_t* state_bytes) {
  return un_plan_bytes_grouped(specs, n_models, in, 1, nullptr, arena_bytes, state_bytes);
}

un_status un_create(const un_model_spec* specs, int32_t n_models, const un_input_spec* in, un_ctx** out) {
  return un_create_grouped(specs, n_models, in, 1, nullptr, out);
}

un_status un_create_grouped(const un_model_spec* specs, int32_t n_models, const un_input_spec* inputs,
                            int32_t n_groups, const int32_t* group_of, un_ctx** out) {
  if (!out) return fail(nullptr, UN_ERR_INVALID, "out is NULL");
  *out = nullptr;
  un_ctx* c = nullptr;
  {
    un_status ps = parse_all(specs, n_models, inputs, n_groups, group_of, &c);
    if (ps != UN_OK) return ps;
  }
  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking);
  if (e != hipSuccess) {
    delete c;
    return fail(nullptr, UN_ERR_DEVICE, std::string("hipStreamCreate: ") + hipGetErrorString(e));
  }
  c->own_stream = c->stream;
  un_status s = plan_and_alloc(c);
  if (s != UN_OK) {
    std::string msg = c->err.empty() ? g_create_error : c->err;
    if (c->base) hipFree(c->base);
    hipStreamDestroy(c->own_stream);
    delete c;
    return fail(nullptr, s, msg);
  }
  std::vector<float> pt;
  for (int i = 0; i < n_models; ++i) {
    init_host(c->models[i], pt);
    s = write_params(c, i, pt.data());
    if (s != UN_OK) break;
  }
  if (s == UN_OK) s = refresh_copies(c);
  if (s == UN_OK && hipStreamSynchronize(c->stream) != hipSuccess) s = UN_ERR_DEVICE;
  if (s != UN_OK) {
    std::string msg = c->err;
    un_destroy(c);
    return fail(nullptr, s, msg);
  }
  *out = c;
  return UN_OK;
}

static un_status load_common(un_ctx* c, int gi, const float* x, const int32_t* y, bool device) {
  Group& g = c->groups[gi];
  const size_t nx = (size_t)g.B * g.in_feat;
  std::vector<int32_t> yh(g.B);
  if (device) {
    HIPCHK(c, hipMemcpyAsync(yh.data(), y, (size_t)g.B * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
  } else {
    memcpy(yh.data(), y, (size_t)g.B * 4);
  }
  for (int b = 0; b < g.B; ++b)
    if (yh[b] < 0 || yh[b] >= g.min_classes)
      return fail(c, UN_ERR_RANGE, "label " + std::to_string(yh[b]) + " at " + std::to_string(b) + " out of range");
  const float* xsrc = x;
  if (!device) {
    HIPCHK(c, hipMemcpyAsync(c->base + g.xstage, x, nx * 4, hipMemcpyHostToDevice, c->stream));
    xsrc = c->at<float>(g.xstage);
  }
  HIPCHK(c, hipMemcpyAsync(c->base + c->ydev + g.lab_shared * 4, yh.data(), (size_t)g.B * 4, hipMemcpyHostToDevice,
                           c->stream));
  HIPCHK(c, launch_load(c->bf16, xsrc, g.B, g.in_c, g.in_h, g.in_w, g.Xin == NONE ? nullptr : c->base + g.Xin,
                        g.XinC == NONE ? nullptr : c->base + g.XinC, g.in_cs, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  g.loaded = true;
  c->labels_per_model = false;
  return UN_OK;
}

un_status un_load_batch(un_ctx* c, const float* x, const int32_t* y) {
  CHECK_CTX(c);
  if (!x || !y) return fail(c, UN_ERR_INVALID, "x or y is NULL");
  if (c->groups.size() != 1) return fail(c, UN_ERR_INVALID, "several input groups: use un_load_group_batch");
  return load_common(c, 0, x, y, false);
}

un_status un_load_batch_device(un_ctx* c, const float* x, const int32_t* y) {
  CHECK_CTX(c);
  if (!x || !y) return fail(c, UN_ERR_INVALID, "x or y is NULL");
  if (c->groups.size() != 1) return fail(c, UN_ERR_INVALID, "several input groups: use un_load_group_batch");
  return load_common(c, 0, x, y, true);
}

un_status un_load_group_batch(un_ctx* c, int32_t g, const float* x, const int32_t* y) {
  CHECK_CTX(c);
  if (!x || !y) return fail(c, UN_ERR_INVALID, "x or y is NULL");
  if (g < 0 || g >= (int)c->groups.size()) return fail(c, UN_ERR_RANGE, "input group out of range");
  return load_common(c, g, x, y, false);
}

// The kernels of one step, in order, on the context's stream.
static hipError_t enqueue_step(un_ctx* c, float lr) {
  for (auto& l : c->fwd) {
    hipError_t e = run_launch(c, l, lr);
    if (e != hipSuccess) return e;
  }
  hipError_t e = run_launch(c, c->ce, lr);
  for (auto& l : c->bwd) {
    if (e != hipSuccess) return e;
    e = run_launch(c, l, lr);
  }
  return e;
}

// The step's launches. Rates: lrs (host, per model) or else lr for every
// model. With an optimizer other than SGD on some model, every model's
// OptHp (rate folded in) goes to the device first and the update kernels
// follow it; otherwise per-model rates go to lr_dev, or lr is passed as is.
static un_status step_common(un_ctx* c, float lr, const float* lrs, float* losses) {
  struct Reset {
    un_ctx* c;
    ~Reset() {
      c->lrv = nullptr;
      c->optp = nullptr;
    }
  } reset{c};
  const size_t n = c->models.size();
  if (c->any_opt) {
    std::vector<OptHp> hp(n);
    for (size_t i = 0; i < n; ++i) {
      const auto& o = c->opts[i];
      const double rate = lrs ? (double)lrs[i] : (double)lr;
      OptHp& h = hp[i];
      h.kind = (float)o.kind;
      h.lr = (float)rate;
      h.eps = (float)o.eps;
      if (o.kind == UN_OPT_MOMENTUM) {
        h.b1 = (float)o.momentum;
      } else if (o.kind == UN_OPT_ADAM) {
        const double t = (double)(o.t + 1);  // this step's count
        h.b1 = (float)o.beta1;
        h.b2 = (float)o.beta2;
        h.c1 = (float)(1.0 - o.beta1);
        h.c2 = (float)(1.0 - o.beta2);
        h.lr = (float)(rate / (1.0 - std::pow(o.beta1, t)));
        h.isb2 = (float)(1.0 / std::sqrt(1.0 - std::pow(o.beta2, t)));
      }
    }
    HIPCHK(c, launch_set_values(c->at<float>(c->opt_dev), (const float*)hp.data(), (int)(n * OPT_FLOATS), c->stream));
    c->optp = c->at<OptHp>(c->opt_dev);
  } else if (lrs) {
    HIPCHK(c, launch_set_values(c->at<float>(c->lr_dev), lrs, (int)n, c->stream));
    c->lrv = c->at<float>(c->lr_dev);
  }
  HIPCHK(c, enqueue_step(c, lr));
  for (size_t i = 0; i < n; ++i)
    if (c->active[i]) ++c->opts[i].t;
  c->stepped = true;
  c->grads_valid = c->keep_grads;
  if (c->profiling && c->recs.size() > 4096) {
    un_status s = drain_profile(c);
    if (s != UN_OK) return s;
  }
  if (losses) {
    HIPCHK(c, hipMemcpyAsync(losses, c->base + c->losses_dev, c->models.size() * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    for (size_t i = 0; i < c->models.size(); ++i)
      if (!c->active[i]) losses[i] = std::nanf("");
  }
  return UN_OK;
}

un_status un_step(un_ctx* c, float lr, float* losses) {
  CHECK_CTX(c);
  if (!c->all_loaded()) return fail(c, UN_ERR_STATE, "un_step before a batch of every input group is loaded");
  if (!std::isfinite(lr)) return fail(c, UN_ERR_INVALID, "lr is not finite");
  return step_common(c, lr, nullptr, losses);
}

un_status un_step_lr(un_ctx* c, const float* lrs, float* losses) {
  CHECK_CTX(c);
  if (!lrs) return fail(c, UN_ERR_INVALID, "lrs is NULL");
  if (!c->all_loaded()) return fail(c, UN_ERR_STATE, "un_step_lr before a batch of every input group is loaded");
  for (size_t i = 0; i < c->models.size(); ++i)
    if (!std::isfinite(lrs[i])) return fail(c, UN_ERR_INVALID, "lr of model " + std::to_string(i) + " is not finite");
  // the rates travel in kernel arguments, ordered before the step on the stream
  return step_common(c, 0.f, lrs, losses);
}

// ---- optimizers -----------------------------------------------------------
// The state allocation mirrors the parameter layout: one momentum / first
// moment and one second moment per parameter, for every model (made once, on
// the first optimizer that needs state; the step's tables are rebuilt to point
// at it).
static size_t state_layout(un_ctx* c) {
  Arena S;
  for (auto& g : c->groups) {
    if (g.cat.empty()) continue;
    g.catS1 = S.take((size_t)g.cat_rows * g.kin_p * 4);
    g.catS1b = S.take((size_t)g.cat_rows * 4);
    g.catS2 = S.take((size_t)g.cat_rows * g.kin_p * 4);
    g.catS2b = S.take((size_t)g.cat_rows * 4);
  }
  for (size_t mi = 0; mi < c->models.size(); ++mi)
    for (auto& b : c->models[mi].blocks) {
      if (b.kind == 2) continue;
      if (b.concat) {
        const Group& g = c->groups[c->models[mi].group];
        const size_t roff = (size_t)c->cat_off[mi];
        b.S1 = g.catS1 + roff * b.ldw * 4;
        b.S2 = g.catS2 + roff * b.ldw * 4;
        b.S1b = g.catS1b + roff * 4;
        b.S2b = g.catS2b + roff * 4;
      } else {
        b.S1 = S.take((size_t)b.rows * b.ldw * 4);
        b.S1b = S.take((size_t)b.rows * 4);
        b.S2 = S.take((size_t)b.rows * b.ldw * 4);
        b.S2b = S.take((size_t)b.rows * 4);
      }
    }
  return S.top;
}

static un_status alloc_state(un_ctx* c) {
  const size_t bytes = state_layout(c);
  char* p = nullptr;
  hipError_t e = hipMalloc((void**)&p, bytes);
  if (e != hipSuccess) return fail(c, UN_ERR_OOM, "optimizer state: hipMalloc of " + std::to_string(bytes) + " bytes failed");
  HIPCHK(c, hipMemsetAsync(p, 0, bytes, c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  c->sbase = p;
  c->sbytes = bytes;
  Tables T;
  build_tables(c, T);
  return install_tables(c, T);
}

// Zero model i's optimizer state.
static un_status clear_state(un_ctx* c, int i) {
  if (!c->sbase) return UN_OK;
  for (auto& b : c->models[i].blocks) {
    if (b.kind == 2) continue;
    HIPCHK(c, hipMemsetAsync(c->sbase + b.S1, 0, (size_t)b.rows * b.ldw * 4, c->stream));
    HIPCHK(c, hipMemsetAsync(c->sbase + b.S2, 0, (size_t)b.rows * b.ldw * 4, c->stream));
    HIPCHK(c, hipMemsetAsync(c->sbase + b.S1b, 0, (size_t)b.rows * 4, c->stream));
    HIPCHK(c, hipMemsetAsync(c->sbase + b.S2b, 0, (size_t)b.rows * 4, c->stream));
  }
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return UN_OK;
}

static int state_tensors(int kind) { return kind == UN_OPT_ADAM ? 2 : kind == UN_OPT_MOMENTUM ? 1 : 0; }

un_status un_set_optimizer(un_ctx* c, int32_t i, const un_optimizer* o) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  if (!o) return fail(c, UN_ERR_INVALID, "optimizer is NULL");
  auto unit = [](float x) { return std::isfinite(x) && x >= 0.f && x < 1.f; };
  if (o->kind != UN_OPT_SGD && o->kind != UN_OPT_MOMENTUM && o->kind != UN_OPT_ADAM)
    return fail(c, UN_ERR_INVALID, "unknown optimizer kind");
  if (o->kind == UN_OPT_MOMENTUM && !unit(o->momentum)) return fail(c, UN_ERR_INVALID, "momentum must be in [0, 1)");
  if (o->kind == UN_OPT_ADAM && (!unit(o->beta1) || !unit(o->beta2) || !std::isfinite(o->eps) || !(o->eps > 0.f)))
    return fail(c, UN_ERR_INVALID, "Adam needs beta1, beta2 in [0, 1) and eps > 0");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  if (o->kind != UN_OPT_SGD && !c->sbase) {
    un_status st = alloc_state(c);
    if (st != UN_OK) return st;
  }
  un_status st = clear_state(c, i);
  if (st != UN_OK) return st;
  un_ctx::Opt& d = c->opts[i];
  d.kind = o->kind;
  d.momentum = o->momentum;
  d.beta1 = o->beta1;
  d.beta2 = o->beta2;
  d.eps = o->eps;
  d.t = 0;
  c->any_opt = false;
  for (auto& x : c->opts) c->any_opt = c->any_opt || x.kind != UN_OPT_SGD;
  return UN_OK;
}

un_status un_get_opt_state(un_ctx* c, int32_t i, float* dst, size_t cap, size_t* n, int64_t* step) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  const int k = state_tensors(c->opts[i].kind);
  const size_t np = c->models[i].n_params;
  if (n) *n = k * np;
  if (step) *step = c->opts[i].t;
  if (!dst || k == 0) return UN_OK;
  if (cap < k * np) return fail(c, UN_ERR_BUFSIZE, "buffer holds " + std::to_string(cap) + " < " + std::to_string(k * np));
  un_status st = read_blocks(c, i, c->sbase, &Block::S1, &Block::S1b, dst);
  if (st == UN_OK && k == 2) st = read_blocks(c, i, c->sbase, &Block::S2, &Block::S2b, dst + np);
  return st;
}

un_status un_set_opt_state(un_ctx* c, int32_t i, const float* src, size_t n, int64_t step) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  const int k = state_tensors(c->opts[i].kind);
  const size_t np = c->models[i].n_params;
  if (n != k * np) return fail(c, UN_ERR_BUFSIZE, "state of this optimizer holds " + std::to_string(k * np) + " floats");
  if (step < 0) return fail(c, UN_ERR_INVALID, "negative step count");
  if (k > 0 && !src) return fail(c, UN_ERR_INVALID, "src is NULL");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  if (k > 0) {
    un_status st = write_blocks(c, i, c->sbase, &Block::S1, &Block::S1b, src);
    if (st == UN_OK && k == 2) st = write_blocks(c, i, c->sbase, &Block::S2, &Block::S2b, src + np);
    if (st != UN_OK) return st;
  }
  c->opts[i].t = step;
  return UN_OK;
}

un_status un_load_labels(un_ctx* c, const int32_t* y) {
  CHECK_CTX(c);
  if (!y) return fail(c, UN_ERR_INVALID, "y is NULL");
  if (!c->all_loaded()) return fail(c, UN_ERR_STATE, "un_load_labels before a batch of every input group is loaded");
  const size_t n = c->models.size();
  size_t off = 0;
  for (size_t i = 0; i < n; ++i) {
    const size_t B = (size_t)c->groups[c->models[i].group].B;
    for (size_t b = 0; b < B; ++b) {
      const int32_t v = y[off + b];
      if (v < 0 || v >= c->models[i].num_classes)
        return fail(c, UN_ERR_RANGE, "label " + std::to_string(v) + " of model " + std::to_string(i) + " at " +
                                         std::to_string(b) + " out of range");
    }
    off += B;
  }
  // the model rows follow the group rows and are laid out in model order, as y
  HIPCHK(c, hipMemcpyAsync(c->base + c->ydev + c->models[0].lab_own * 4, y, off * 4, hipMemcpyHostToDevice,
                           c->stream));
  HIPCHK(c, hipStreamSynchronize(c->stream));
  c->labels_per_model = true;
  return UN_OK;
}

un_status un_set_active(un_ctx* c, const uint8_t* mask) {
  CHECK_CTX(c);
  if (!mask) return fail(c, UN_ERR_INVALID, "mask is NULL");
  std::vector<char> act(c->models.size());
  bool any = false;
  for (size_t i = 0; i < act.size(); ++i) {
    act[i] = mask[i] != 0;
    any = any || act[i];
  }
  if (!any) return fail(c, UN_ERR_INVALID, "no active model");
  if (act == c->active) return UN_OK;
  HIPCHK(c, hipStreamSynchronize(c->stream));  // the current tables are no longer in use
  const std::vector<char> before = c->active;
  c->active = act;
  Tables T;
  build_tables(c, T);
  un_status st = install_tables(c, T);
  if (st != UN_OK) {
    c->active = before;
    return st;
  }
  // Models that sat out some steps kept their transposed weight copy in the
  // buffer of that time; rewrite every model's current copies from the master.
  st = refresh_copies(c);
  if (st != UN_OK) return st;
  HIPCHK(c, hipStreamSynchronize(c->stream));
  c->grads_valid = false;
  return UN_OK;
}

// Device address of the scratch array on the context's device (looked up with
// that device current, the first time only).
static un_status scratch_on(un_ctx* c, char** out) {
  if (c->device < 0 || c->device >= MAX_DEVICES) return fail(c, UN_ERR_UNSUPPORTED, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[c->device]) {
    int cur = 0;
    HIPCHK(c, hipGetDevice(&cur));
    if (cur != c->device) HIPCHK(c, hipSetDevice(c->device));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != c->device) HIPCHK(c, hipSetDevice(cur));
    HIPCHK(c, e);
    if (!p) return fail(c, UN_ERR_DEVICE, "hipGetSymbolAddress returned no address for the scratch array");
    g_scratch_ptr[c->device] = (char*)p;
  }
  *out = g_scratch_ptr[c->device];
  return UN_OK;
}

un_status un_step_scratch(un_ctx* c, float lr, float* losses) {
  CHECK_CTX(c);
  if (!c->all_loaded()) return fail(c, UN_ERR_STATE, "un_step_scratch before a batch of every input group is loaded");
  if (!std::isfinite(lr)) return fail(c, UN_ERR_INVALID, "lr is not finite");
  if (c->ws_bytes > UN_SCRATCH_BYTES)
    return fail(c, UN_ERR_UNSUPPORTED, "this context's step workspace (" + std::to_string(c->ws_bytes) +
                                           " bytes) exceeds the library's static scratch (" +
                                           std::to_string(UN_SCRATCH_BYTES) + " bytes); use un_step");
  char* ptr = nullptr;
  un_status st = scratch_on(c, &ptr);
  if (st != UN_OK) return st;
  // every workspace pointer of the tables moves by the same offset into the scratch array
  c->wsoff = (int64_t)(ptr - (c->base + c->ws_lo));
  st = step_common(c, lr, nullptr, losses);
  c->wsoff = 0;
  return st;
}

un_status un_set_stream(un_ctx* c, void* stream) {
  CHECK_CTX(c);
  HIPCHK(c, hipStreamSynchronize(c->stream));  // the work enqueued so far completes first
  c->stream = stream ? (hipStream_t)stream : c->own_stream;
  c->graph_valid = false;
  return UN_OK;
}

un_status un_graph_capture(un_ctx* c, float lr) {
  CHECK_CTX(c);
  if (!c->all_loaded()) return fail(c, UN_ERR_STATE, "un_graph_capture before a batch of every input group is loaded");
  if (!std::isfinite(lr)) return fail(c, UN_ERR_INVALID, "lr is not finite");
  if (c->any_opt)
    return fail(c, UN_ERR_UNSUPPORTED, "a model has a momentum / Adam optimizer (its hyper-parameters change every step)");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  if (c->gexec) hipGraphExecDestroy(c->gexec);
  if (c->graph) hipGraphDestroy(c->graph);
  c->gexec = nullptr;
  c->graph = nullptr;
  c->graph_valid = false;
  const bool prof = c->profiling;
  c->profiling = false;  // no event records inside the graph
  hipError_t e = hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal);
  hipError_t le = e == hipSuccess ? enqueue_step(c, lr) : hipSuccess;
  hipGraph_t g = nullptr;
  if (e == hipSuccess) e = hipStreamEndCapture(c->stream, &g);
  c->profiling = prof;
  if (e == hipSuccess) e = le;
  if (e == hipSuccess) e = hipGraphInstantiate(&c->gexec, g, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    if (g) hipGraphDestroy(g);
    c->gexec = nullptr;
    c->poisoned = true;
    return fail(c, UN_ERR_DEVICE, std::string("step capture: ") + hipGetErrorString(e));
  }
  c->graph = g;
  c->graph_valid = true;
  c->graph_keep = c->keep_grads;
  c->graph_labels = c->labels_per_model;
  return UN_OK;
}

un_status un_graph_step(un_ctx* c, float* losses) {
  CHECK_CTX(c);
  if (!c->graph_valid || c->graph_keep != c->keep_grads || c->graph_labels != c->labels_per_model || c->any_opt)
    return fail(c, UN_ERR_STATE, "no captured step for the current configuration (un_graph_capture)");
  HIPCHK(c, hipGraphLaunch(c->gexec, c->stream));
  for (size_t i = 0; i < c->models.size(); ++i)
    if (c->active[i]) ++c->opts[i].t;
  c->stepped = true;
  c->grads_valid = c->keep_grads;
  if (losses) {
    HIPCHK(c, hipMemcpyAsync(losses, c->base + c->losses_dev, c->models.size() * 4, hipMemcpyDeviceToHost, c->stream));
    HIPCHK(c, hipStreamSynchronize(c->stream));
    for (size_t i = 0; i < c->models.size(); ++i)
      if (!c->active[i]) losses[i] = std::nanf("");
  }
  return UN_OK;
}

un_status un_param_count(const un_ctx* c, int32_t i, size_t* n) {
  if (!c || !n) return fail(const_cast<un_ctx*>(c), UN_ERR_INVALID, "NULL argument");
  if (i < 0 || i >= (int)c->models.size()) return fail(const_cast<un_ctx*>(c), UN_ERR_RANGE, "model index out of range");
  *n = c->models[i].n_params;
  return UN_OK;
}

un_status un_get_params(un_ctx* c, int32_t i, float* dst, size_t cap, size_t* n) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  const size_t np = c->models[i].n_params;
  if (n) *n = np;
  if (!dst) return UN_OK;
  if (cap < np) return fail(c, UN_ERR_BUFSIZE, "buffer holds " + std::to_string(cap) + " < " + std::to_string(np));
  return read_tensors(c, i, false, dst);
}

un_status un_get_grads(un_ctx* c, int32_t i, float* dst, size_t cap, size_t* n) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  const size_t np = c->models[i].n_params;
  if (n) *n = np;
  if (!dst) return UN_OK;
  if (!c->stepped) return fail(c, UN_ERR_STATE, "no step has run yet");
  if (!c->grads_valid) return fail(c, UN_ERR_STATE, "the last step did not keep gradients (see un_keep_grads)");
  if (!c->active[i]) return fail(c, UN_ERR_STATE, "model " + std::to_string(i) + " was not active in the last step");
  if (cap < np) return fail(c, UN_ERR_BUFSIZE, "buffer too small");
  return read_tensors(c, i, true, dst);
}

un_status un_set_params(un_ctx* c, int32_t i, const float* src, size_t n) {
  CHECK_CTX(c);
  if (i < 0 || i >= (int)c->models.size()) return fail(c, UN_ERR_RANGE, "model index out of range");
  if (!src) return fail(c, UN_ERR_INVALID, "src is NULL");
  if (n != c->models[i].n_params) return fail(c, UN_ERR_BUFSIZE, "element count mismatch");
  HIPCHK(c, hipStreamSynchronize(c->stream));
  un_status s = write_params(c, i, src);
  if (s != UN_OK) return s;
  s = refresh_copies(c, i);
  if (s != UN_OK) return s;
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return UN_OK;
}

un_status un_keep_grads(un_ctx* c, int32_t enable) {
  CHECK_CTX(c);
  c->keep_grads = enable != 0;
  return UN_OK;
}

un_status un_arena_bytes(const un_ctx* c, size_t* bytes) {
  if (!c || !bytes) return fail(const_cast<un_ctx*>(c), UN_ERR_INVALID, "NULL argument");
  *bytes = c->bytes;
  return UN_OK;
}

un_status un_sync(un_ctx* c) {
  CHECK_CTX(c);
  HIPCHK(c, hipStreamSynchronize(c->stream));
  return UN_OK;
}

un_status un_get_stream(const un_ctx* c, void** s) {
  if (!c || !s) return fail(const_cast<un_ctx*>(c), UN_ERR_INVALID, "NULL argument");
  *s = (void*)c->stream;
  return UN_OK;
}

un_status un_profile_enable(un_ctx* c, int32_t enable) {
  CHECK_CTX(c);
  un_status s = drain_profile(c);
  if (s != UN_OK) return s;
  c->profiling = enable != 0;
  if (c->profiling)
    for (int k = 0; k < UN_K_COUNT; ++k) {
      c->prof_ms[k] = 0;
      c->prof_n[k] = 0;
    }
  return UN_OK;
}

un_status un_profile_read(un_ctx* c, int32_t kc, double* ms, int64_t* n) {
  CHECK_CTX(c);
  if (kc < 0 || kc >= UN_K_COUNT) return fail(c, UN_ERR_RANGE, "kernel class out of range");
  un_status s = drain_profile(c);
  if (s != UN_OK) return s;
  if (ms) *ms = c->prof_ms[kc];
  if (n) *n = c->prof_n[kc];
  return UN_OK;
}

void un_destroy(un_ctx* c) {
  if (!c) return;
  if (c->stream) hipStreamSynchronize(c->stream);
  for (auto& r : c->recs) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  for (auto e : c->free_events) hipEventDestroy(e);
  if (c->gexec) hipGraphExecDestroy(c->gexec);
  if (c->graph) hipGraphDestroy(c->graph);
  if (c->base) hipFree(c->base);
  if (c->sbase) hipFree(c->sbase);
  if (c->own_stream) hipStreamDestroy(c->own_stream);
  delete c;
}

const char* un_last_error(const un_ctx* c) {
  if (!c) return g_create_error.c_str();
  return c->err.c_str();
}

}  // extern "C"
