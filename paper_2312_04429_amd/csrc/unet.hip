// UNet handle, execution plan and the K-skipped DDIM loop (host side).
//
// nv_unet_create packs the canonical float32 weight blob into device layouts
// (3x3 conv weights [Cout][ky][kx][Cin] float16, linear [out][in] float16,
// self-attention q|k|v and cross-attention k|v concatenated, GEGLU rows
// interleaved in groups of 16, every ResBlock's time projection stacked into
// one matrix; norms and biases float32).
//
// A plan is the ordered list of kernel launches of one UNet evaluation for up
// to R rows (2 per sample: unconditional, conditional), with every
// activation placed in the caller's workspace by a first-fit arena over
// buffer lifetimes.  The same plan runs with fewer active rows: all
// activations are row-major with rows outermost.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <map>
#include <memory>
#include <numeric>
#include <string>
#include <vector>

#include "attention.h"
#include "common.h"
#include "gemm.h"
#include "ops.h"
#include "trace.h"

namespace nv {

static thread_local std::string g_err;
void set_error(const std::string& m) { g_err = m; }
void clear_error() { g_err.clear(); }

namespace {

struct ParamInfo {
  std::string name;
  std::vector<int64_t> shape;
  int64_t offset = 0;
  int64_t numel() const {
    int64_t n = 1;
    for (auto s : shape) n *= s;
    return n;
  }
};

// Transformer LayerNorms can be folded into the products that consume them
// (self-attention q|k|v, cross-attention q, GEGLU) when the channel count is
// whole 64-deep k tiles, as the streamed GEMM requires:
//   LN(x) W^T = rstd * (x (gamma W)^T - mean * sum_k gamma_k W[n][k]) + beta W^T.
// A call folds them when the LayerNorm's input is at most LN_FOLD_MAX_ELEMS
// values (8192 tokens of 320 channels: batch-1 shapes, where the products are
// latency-bound and the saved launch pays); on larger inputs the row
// statistics' extra LDS reads cost more than the launch saves.
inline bool ln_folded(int ch) { return ch % 64 == 0; }
constexpr int64_t LN_FOLD_MAX_ELEMS = 8192 * 320;

int heads_for(const nv_unet_config& c, int ch) {
  return c.n_heads > 0 ? c.n_heads : ch / c.head_dim;
}

// Canonical parameter order (documented in nv.h).
void enumerate_params(const nv_unet_config& c, std::vector<ParamInfo>& out) {
  out.clear();
  const int c0 = c.ch[0], td = 4 * c0, L = c.n_levels;
  auto add = [&](const std::string& n, std::vector<int64_t> s) { out.push_back({n, s, 0}); };
  auto lin = [&](const std::string& n, int o, int i, bool bias = true) {
    add(n + ".w", {o, i});
    if (bias) add(n + ".b", {o});
  };
  auto conv = [&](const std::string& n, int o, int i) {
    add(n + ".w", {o, i, 3, 3});
    add(n + ".b", {o});
  };
  auto norm = [&](const std::string& n, int ch) {
    add(n + ".g", {ch});
    add(n + ".b", {ch});
  };
  auto res = [&](const std::string& n, int cin, int cout) {
    norm(n + ".gn1", cin);
    conv(n + ".conv1", cout, cin);
    lin(n + ".temb", cout, td);
    norm(n + ".gn2", cout);
    conv(n + ".conv2", cout, cout);
    if (cin != cout) lin(n + ".skip", cout, cin);
  };
  auto tr = [&](const std::string& n, int ch, int depth) {
    norm(n + ".gn", ch);
    lin(n + ".proj_in", ch, ch);
    for (int j = 0; j < depth; ++j) {
      const std::string b = n + ".blk" + std::to_string(j);
      norm(b + ".ln1", ch);
      lin(b + ".attn1.q", ch, ch, false);
      lin(b + ".attn1.k", ch, ch, false);
      lin(b + ".attn1.v", ch, ch, false);
      lin(b + ".attn1.o", ch, ch);
      norm(b + ".ln2", ch);
      lin(b + ".attn2.q", ch, ch, false);
      lin(b + ".attn2.k", ch, c.ctx_dim, false);
      lin(b + ".attn2.v", ch, c.ctx_dim, false);
      lin(b + ".attn2.o", ch, ch);
      norm(b + ".ln3", ch);
      lin(b + ".ff1", 8 * ch, ch);
      lin(b + ".ff2", ch, 4 * ch);
    }
    lin(n + ".proj_out", ch, ch);
  };
  lin("time.l1", td, c0);
  lin("time.l2", td, td);
  conv("conv_in", c0, c.in_ch);
  std::vector<int> skips{c0};
  int cur = c0;
  for (int lv = 0; lv < L; ++lv) {
    const int co = c.ch[lv];
    for (int r = 0; r < c.n_res; ++r) {
      res("down" + std::to_string(lv) + ".res" + std::to_string(r), cur, co);
      cur = co;
      if (c.depth[lv] > 0)
        tr("down" + std::to_string(lv) + ".attn" + std::to_string(r), cur, c.depth[lv]);
      skips.push_back(cur);
    }
    if (lv < L - 1) {
      conv("down" + std::to_string(lv) + ".ds", cur, cur);
      skips.push_back(cur);
    }
  }
  res("mid.res0", cur, cur);
  if (c.mid_depth > 0) tr("mid.attn", cur, c.mid_depth);
  res("mid.res1", cur, cur);
  for (int lv = L - 1; lv >= 0; --lv) {
    const int co = c.ch[lv];
    for (int r = 0; r < c.n_res + 1; ++r) {
      const int sk = skips.back();
      skips.pop_back();
      res("up" + std::to_string(lv) + ".res" + std::to_string(r), cur + sk, co);
      cur = co;
      if (c.depth[lv] > 0)
        tr("up" + std::to_string(lv) + ".attn" + std::to_string(r), cur, c.depth[lv]);
    }
    if (lv > 0) conv("up" + std::to_string(lv) + ".us", cur, cur);
  }
  norm("out.gn", cur);
  conv("conv_out", c.out_ch, cur);
  int64_t off = 0;
  for (auto& p : out) {
    p.offset = off;
    off += p.numel();
  }
}

bool validate_cfg(const nv_unet_config* c, std::string* why) {
  auto fail = [&](const std::string& m) {
    *why = m;
    return false;
  };
  if (!c) return fail("null config");
  if (c->in_ch < 1 || c->in_ch > 16 || c->out_ch < 1 || c->out_ch > 16)
    return fail("in_ch/out_ch must be in [1, 16]");
  if (c->n_levels < 1 || c->n_levels > 4) return fail("n_levels must be in [1, 4]");
  if (c->n_res < 1 || c->n_res > 8) return fail("n_res must be in [1, 8]");
  if (c->gn_groups < 4 || c->gn_groups > 256 || 256 % c->gn_groups)
    return fail("gn_groups must be a power of two in [4, 256]");
  const int f = 1 << (c->n_levels - 1);
  if (c->H < f || c->W < f || c->H % f || c->W % f)
    return fail("H and W must be divisible by 2^(n_levels-1)");
  if (c->ctx_len < 1 || c->ctx_dim < 8 || c->ctx_dim % 8) return fail("bad context shape");
  if (!(c->gn_eps > 0) || !(c->ln_eps > 0)) return fail("eps must be > 0");
  if ((size_t)c->ch[0] * c->in_ch * 36 + (size_t)c->ch[0] * 4 > 160 * 1024)
    return fail("conv_in weights must fit in LDS (ch[0] * in_ch * 9 floats)");
  if (c->pooled_dim != 0 && c->pooled_dim != 4 * c->ch[0])
    return fail("pooled_dim must be 0 or 4*ch[0]");
  for (int l = 0; l < c->n_levels; ++l) {
    const int ch = c->ch[l];
    if (ch < 32 || ch % 32 || ch % c->gn_groups || ch > 2048)
      return fail("channels must be multiples of 32 and of gn_groups, at most 2048");
    if (c->depth[l] < 0) return fail("depth must be >= 0");
  }
  if (c->mid_depth < 0) return fail("mid_depth must be >= 0");
  // attention head dims and concatenated channel counts
  std::vector<int> skips{c->ch[0]};
  int cur = c->ch[0];
  auto check_tr = [&](int ch) -> bool {
    if (c->n_heads <= 0 && c->head_dim <= 0) return false;
    const int h = heads_for(*c, ch);
    if (h < 1 || ch % h) return false;
    return attn_supported(ch / h);
  };
  for (int l = 0; l < c->n_levels; ++l) {
    for (int r = 0; r < c->n_res; ++r) {
      cur = c->ch[l];
      skips.push_back(cur);
    }
    if (c->depth[l] > 0 && !check_tr(c->ch[l])) return fail("unsupported head dim");
    if (l < c->n_levels - 1) skips.push_back(cur);
  }
  if (c->mid_depth > 0 && !check_tr(cur)) return fail("unsupported head dim (mid)");
  for (int l = c->n_levels - 1; l >= 0; --l)
    for (int r = 0; r < c->n_res + 1; ++r) {
      const int sk = skips.back();
      skips.pop_back();
      const int cin = cur + sk;
      if (cin % c->gn_groups) return fail("concatenated channels must be divisible by gn_groups");
      if (cin == c->ch[l]) return fail("concatenated input equal to output width is unsupported");
      cur = c->ch[l];
    }
  return true;
}

// ---------------------------------------------------------------- weights
struct Lin {
  const _Float16* w = nullptr;
  const float* b = nullptr;
  int out = 0, in = 0;
};
struct Norm {
  const float* g = nullptr;
  const float* b = nullptr;
};

// Execution-time context of one UNet evaluation.
struct RunCtx {
  char* ws;
  int R;             // active rows
  hipStream_t s;
  const float* x;    // float32 latent [samples][Cin][H][W]
  StepArgs st;
  float* partial;    // split-K scratch
  size_t partial_bytes;
  int nsteps = 0;    // grid steps N of the call's schedule
};

inline hipError_t gemm_run(GemmArgs g, const RunCtx& c) {
  g.partial = c.partial;
  g.partial_bytes = c.partial_bytes;
  return gemm_launch(g, c.s);
}
using Op = std::function<hipError_t(const RunCtx&)>;

struct Arena {
  std::vector<std::pair<size_t, size_t>> free_;  // (off, size)
  size_t top = 0;
  size_t alloc(size_t bytes) {
    bytes = align_up(std::max<size_t>(bytes, 1), 256);
    for (size_t i = 0; i < free_.size(); ++i) {
      if (free_[i].second >= bytes) {
        const size_t off = free_[i].first;
        free_[i].first += bytes;
        free_[i].second -= bytes;
        if (free_[i].second == 0) free_.erase(free_.begin() + i);
        return off;
      }
    }
    const size_t off = top;
    top += bytes;
    return off;
  }
  void release(size_t off, size_t bytes) {
    bytes = align_up(std::max<size_t>(bytes, 1), 256);
    free_.push_back({off, bytes});
    std::sort(free_.begin(), free_.end());
    std::vector<std::pair<size_t, size_t>> m;
    for (auto& f : free_) {
      if (!m.empty() && m.back().first + m.back().second == f.first)
        m.back().second += f.second;
      else
        m.push_back(f);
    }
    if (!m.empty() && m.back().first + m.back().second == top) {
      top = m.back().first;
      m.pop_back();
    }
    free_ = m;
  }
};

struct Ten {
  int id = -1;
  size_t off = 0;
  int HW = 0, C = 0;
};

constexpr size_t SPLITK_BYTES = 32u << 20;  // float32 split-K partials

struct Plan {
  int Rmax = 0;
  std::vector<Op> pre;   // once per call (context projections)
  std::vector<Op> step;  // one UNet evaluation
  size_t bytes = 0;
  // fixed regions
  size_t x_work = 0, eps = 0, ts = 0, at = 0, ap = 0, ctx = 0, pooled = 0, tproj = 0;
  size_t gnpart = 0, splitk = 0;
  size_t stepdev = 0;  // int32 [2][MAX_SAMPLES]: current grid step and caller index per sample
  size_t ttab = 0;     // float32 [MAX_GRID_STEPS][temb_total]: ResBlock time projections per grid step
};

// A schedule has N <= T / 2 <= 512 grid steps.
constexpr int MAX_GRID_STEPS = 512;

// What a captured denoise step depends on besides the active rows: the plan
// (its buffer offsets), the workspace and the update's constants.
struct GraphKey {
  const Plan* plan = nullptr;
  const char* ws = nullptr;
  float guidance = 0.f, eta = 0.f;
  const float* z = nullptr;
  int N = 0;
  bool operator==(const GraphKey& o) const {
    return plan == o.plan && ws == o.ws && guidance == o.guidance && eta == o.eta && z == o.z &&
           N == o.N;
  }
};

}  // namespace
}  // namespace nv

struct nv_unet {
  nv_unet_config cfg;
  std::vector<nv::ParamInfo> params;
  std::map<std::string, const _Float16*> w16;
  std::map<std::string, const float*> w32;
  _Float16* d16 = nullptr;
  float* d32 = nullptr;
  int temb_total = 0;                       // sum of ResBlock widths
  std::map<std::string, int> temb_off;      // ResBlock name -> column offset
  std::map<int, std::unique_ptr<nv::Plan>> plans;
  // Captured denoise steps (HIP graphs), one per active row count, valid for
  // gkey; replaying one costs about half the dispatch time of launching its
  // kernels one by one.
  bool use_graphs = true;
  hipStream_t capture_stream = nullptr;
  nv::GraphKey gkey;
  std::map<int, hipGraphExec_t> graphs;
  void drop_graphs() {
    for (auto& kv : graphs) (void)hipGraphExecDestroy(kv.second);
    graphs.clear();
  }
};

namespace nv {
namespace {

class Builder {
 public:
  Builder(nv_unet* net, Plan* p, int Rmax) : net_(net), P(p), Rmax_(Rmax) {}

  Ten alloc(int HW, int C, int esize = 2) {
    Ten t;
    t.id = (int)sizes_.size();
    t.HW = HW;
    t.C = C;
    const size_t bytes = (size_t)Rmax_ * HW * C * esize;
    t.off = arena_.alloc(bytes);
    sizes_.push_back(bytes);
    refs_.push_back(1);
    offs_.push_back(t.off);
    return t;
  }
  size_t fixed(size_t bytes) { return arena_.alloc(bytes); }
  void hold(const Ten& t) { refs_[t.id]++; }
  void drop(const Ten& t) {
    if (--refs_[t.id] == 0) arena_.release(offs_[t.id], sizes_[t.id]);
  }
  size_t peak() const { return arena_.top_peak; }

  const _Float16* W16(const std::string& n) {
    auto it = net_->w16.find(n);
    if (it == net_->w16.end()) throw std::runtime_error("missing weight " + n);
    return it->second;
  }
  const float* W32(const std::string& n) {
    auto it = net_->w32.find(n);
    if (it == net_->w32.end()) throw std::runtime_error("missing weight " + n);
    return it->second;
  }

  nv_unet* net_;
  Plan* P;
  int Rmax_;
  struct TrackedArena : Arena {
    size_t top_peak = 0;
    size_t alloc(size_t b) {
      const size_t o = Arena::alloc(b);
      top_peak = std::max(top_peak, top);
      return o;
    }
  } arena_;
  std::vector<size_t> sizes_, offs_;
  std::vector<int> refs_;
};

inline _Float16* H16(const RunCtx& c, size_t off) { return (_Float16*)(c.ws + off); }
inline float* F32(const RunCtx& c, size_t off) { return (float*)(c.ws + off); }

// GEMM op helpers --------------------------------------------------------
GemmArgs dense_args(int N, int K, const _Float16* w, const float* bias) {
  GemmArgs g{};
  g.N = N;
  g.K = K;
  g.w = w;
  g.ldw = K;
  g.bias = bias;
  g.C1 = K;
  g.lda1 = K;
  g.rows_div = 1;
  return g;
}

void emit_gn(Builder& B, std::vector<Op>& ops, const Ten& x1, const Ten* x2, const std::string& n,
             bool silu, const Ten& out) {
  const auto& cfg = B.net_->cfg;
  const float* g = B.W32(n + ".g");
  const float* b = B.W32(n + ".b");
  const size_t o1 = x1.off, o2 = x2 ? x2->off : 0, oo = out.off;
  const size_t gp = B.P->gnpart;
  const int part_chunks = (int)ceil_div(B.net_->cfg.H * B.net_->cfg.W, 8);
  const int C1 = x1.C, C2 = x2 ? x2->C : 0, HW = x1.HW, G = cfg.gn_groups;
  const float eps = cfg.gn_eps;
  const bool has2 = x2 != nullptr;
  ops.push_back([=](const RunCtx& c) {
    GnArgs a{};
    a.src1 = H16(c, o1);
    a.src2 = has2 ? H16(c, o2) : nullptr;
    a.C1 = C1;
    a.C2 = C2;
    a.HW = HW;
    a.G = G;
    a.eps = eps;
    a.gamma = g;
    a.beta = b;
    a.silu = silu;
    a.part = F32(c, gp);
    a.part_chunks = part_chunks;
    a.out = H16(c, oo);
    return gn_launch(a, c.R, c.s);
  });
}

struct ConvSpec {
  int Hin, Win, Ho, Wo, stride, upsample;
};

void emit_conv(Builder& B, std::vector<Op>& ops, const Ten& x1, const Ten* x2,
               const std::string& n, int cout, ConvSpec cs, const Ten& out, const Ten* residual,
               int temb_off, bool out_f32 = false, size_t out_off_override = 0) {
  const _Float16* w = B.W16(n + ".w");
  const float* bias = B.W32(n + ".b");
  const size_t o1 = x1.off, o2 = x2 ? x2->off : 0;
  const size_t oo = out_f32 ? out_off_override : out.off;
  const size_t ores = residual ? residual->off : 0;
  const bool has2 = x2 != nullptr, hasr = residual != nullptr;
  const int C1 = x1.C, C2 = x2 ? x2->C : 0;
  const size_t tproj = B.P->tproj;
  const int ttot = B.net_->temb_total;
  ops.push_back([=](const RunCtx& c) {
    GemmArgs g{};
    g.M = (int64_t)c.R * cs.Ho * cs.Wo;
    g.N = cout;
    g.K = 9 * (C1 + C2);
    g.src1 = H16(c, o1);
    g.src2 = has2 ? H16(c, o2) : nullptr;
    g.C1 = C1;
    g.C2 = C2;
    g.conv = 1;
    g.Hin = cs.Hin;
    g.Win = cs.Win;
    g.Ho = cs.Ho;
    g.Wo = cs.Wo;
    g.stride = cs.stride;
    g.upsample = cs.upsample;
    g.w = w;
    g.ldw = g.K;
    g.bias = bias;
    g.rows_div = (int64_t)cs.Ho * cs.Wo;
    if (temb_off >= 0) {
      g.rowvec = F32(c, tproj) + temb_off;
      g.ld_rowvec = ttot;
    }
    if (hasr) {
      g.residual = H16(c, ores);
      g.ld_res = cout;
    }
    g.out = c.ws + oo;
    g.ldo = cout;
    g.out_f32 = out_f32;
    return gemm_run(g, c);
  });
}

// y[M][N] = x[M][K] W^T (+bias) (+residual) ; x may be a 2-source concat
// A LayerNorm folded into the product that consumes it: used by a call whose
// rows (R * HW) are at most max_rows, which then reads the LayerNorm's input.
struct LnFold {
  const _Float16* w = nullptr;  // gamma-scaled weights
  const float* c1 = nullptr;    // row sums of w
  const float* c2 = nullptr;    // beta . W (+ the layer's bias)
  size_t x_off = 0;             // the LayerNorm's input
  float eps = 0.f;
  int64_t max_rows = -1;        // -1: never folded
  bool on(int64_t rows) const { return rows <= max_rows; }
  void apply(GemmArgs& g, const RunCtx& c) const {
    g.w = w;
    g.bias = c2;
    g.ln_c1 = c1;
    g.ln_eps = eps;
    g.src1 = H16(c, x_off);
  }
};

void emit_linear(Builder& B, std::vector<Op>& ops, const Ten& x1, const Ten* x2,
                 const _Float16* w, const float* bias, int N, const Ten& out, const Ten* residual,
                 bool geglu = false, const LnFold& lf = LnFold{}) {
  const size_t o1 = x1.off, o2 = x2 ? x2->off : 0, oo = out.off;
  const size_t ores = residual ? residual->off : 0;
  const bool has2 = x2 != nullptr, hasr = residual != nullptr;
  const int C1 = x1.C, C2 = x2 ? x2->C : 0, HW = x1.HW, ldo = out.C;
  ops.push_back([=](const RunCtx& c) {
    GemmArgs g = dense_args(N, C1 + C2, w, bias);
    g.M = (int64_t)c.R * HW;
    g.src1 = H16(c, o1);
    g.C1 = C1;
    g.lda1 = C1;
    if (has2) {
      g.src2 = H16(c, o2);
      g.C2 = C2;
      g.lda2 = C2;
    }
    if (hasr) {
      g.residual = H16(c, ores);
      g.ld_res = ldo;
    }
    g.geglu = geglu;
    if (lf.on(g.M)) lf.apply(g, c);
    g.out = c.ws + oo;
    g.ldo = ldo;
    return gemm_run(g, c);
  });
}

Ten build_res(Builder& B, std::vector<Op>& ops, const Ten& x1, const Ten* x2,
              const std::string& n, int cout, int H, int W) {
  const int cin = x1.C + (x2 ? x2->C : 0);
  const int HW = H * W;
  Ten a1 = B.alloc(HW, cin);
  emit_gn(B, ops, x1, x2, n + ".gn1", true, a1);
  Ten h = B.alloc(HW, cout);
  const int toff = B.net_->temb_off.at(n);
  emit_conv(B, ops, a1, nullptr, n + ".conv1", cout, {H, W, H, W, 1, 0}, h, nullptr, toff);
  B.drop(a1);
  Ten a2 = B.alloc(HW, cout);
  emit_gn(B, ops, h, nullptr, n + ".gn2", true, a2);
  B.drop(h);
  Ten sk;
  bool own_sk = false;
  if (cin != cout) {
    sk = B.alloc(HW, cout);
    own_sk = true;
    emit_linear(B, ops, x1, x2, B.W16(n + ".skip.w"), B.W32(n + ".skip.b"), cout, sk, nullptr);
  } else {
    sk = x1;
  }
  Ten out = B.alloc(HW, cout);
  emit_conv(B, ops, a2, nullptr, n + ".conv2", cout, {H, W, H, W, 1, 0}, out, &sk, -1);
  B.drop(a2);
  if (own_sk) B.drop(sk);
  return out;
}

struct KvRef {
  size_t off;
};

Ten build_tr(Builder& B, std::vector<Op>& ops, const Ten& x, const std::string& n, int depth,
             int H, int W, const std::map<std::string, size_t>& kv_regions) {
  const auto& cfg = B.net_->cfg;
  const int C = x.C, HW = H * W;
  const int heads = heads_for(cfg, C), dh = C / heads;
  const int Lc = cfg.ctx_len;
  const float scale = 1.0f / std::sqrt((float)dh);
  Ten g = B.alloc(HW, C);
  emit_gn(B, ops, x, nullptr, n + ".gn", false, g);
  Ten h = B.alloc(HW, C);
  emit_linear(B, ops, g, nullptr, B.W16(n + ".proj_in.w"), B.W32(n + ".proj_in.b"), C, h, nullptr);
  B.drop(g);
  for (int j = 0; j < depth; ++j) {
    const std::string b = n + ".blk" + std::to_string(j);
    // LayerNorm: its own kernel into t, or, for a call whose LayerNorm input
    // is small (at most LN_FOLD_MAX_ELEMS values) and channels that suit the
    // streamed kernel, folded into the product that consumes it (weights
    // packed both ways)
    const int64_t fold_rows = ln_folded(C) ? LN_FOLD_MAX_ELEMS / C : -1;
    const float eps = cfg.ln_eps;
    auto emit_ln = [&](const char* ln, Ten& t) {
      t = B.alloc(HW, C);
      const size_t xi = h.off, to = t.off;
      const float* lg = B.W32(b + ln + ".g");
      const float* lb = B.W32(b + ln + ".b");
      ops.push_back([=](const RunCtx& c) {
        const int64_t rows = (int64_t)c.R * HW;
        if (rows <= fold_rows) return hipSuccess;  // folded into the product
        return layernorm_launch(H16(c, xi), lg, lb, H16(c, to), rows, C, eps, c.s);
      });
    };
    auto fold_of = [&](const std::string& wname, const std::string& cname) {
      LnFold f;
      if (fold_rows < 0) return f;
      f.w = B.W16(wname);
      f.c1 = B.W32(cname + ".c1");
      f.c2 = B.W32(cname + ".c2");
      f.x_off = h.off;
      f.eps = eps;
      f.max_rows = fold_rows;
      return f;
    };
    // self-attention
    Ten t;
    emit_ln(".ln1", t);
    // Q|K as token rows, V written transposed (channel rows, Rmax*HW tokens
    // each) so the attention kernel reads both K and V^T tiles as rows
    Ten qk = B.alloc(HW, 2 * C);
    Ten vt = B.alloc(HW, C);
    {
      const _Float16* w = B.W16(b + ".attn1.qkv.w");
      const LnFold lf = fold_of(b + ".attn1.qkv.wln", b + ".attn1.qkv");
      const size_t xi = t.off, qko = qk.off, vto = vt.off;
      const int64_t vld = (int64_t)B.Rmax_ * HW;
      ops.push_back([=](const RunCtx& c) {
        GemmArgs g = dense_args(3 * C, C, w, nullptr);
        g.M = (int64_t)c.R * HW;
        g.src1 = H16(c, xi);
        if (lf.on(g.M)) lf.apply(g, c);
        g.out = H16(c, qko);
        g.ldo = 2 * C;
        g.vt = H16(c, vto);
        g.vt_col0 = 2 * C;
        g.vt_ld = vld;
        g.vt_div = HW;
        g.vt_stride = HW;
        return gemm_run(g, c);
      });
    }
    B.drop(t);
    Ten a = B.alloc(HW, C);
    {
      const size_t qo = qk.off, vto = vt.off, ao = a.off;
      const int64_t vld = (int64_t)B.Rmax_ * HW;
      ops.push_back([=](const RunCtx& c) {
        AttnArgs at{};
        at.q = H16(c, qo);
        at.k = H16(c, qo) + C;
        at.vt = H16(c, vto);
        at.o = H16(c, ao);
        at.ldq = at.ldk = 2 * C;
        at.ldo = C;
        at.vt_ld = vld;
        at.vt_row = HW;
        at.rows = c.R;
        at.S = HW;
        at.L = HW;
        at.heads = heads;
        at.dh = dh;
        at.scale = scale;
        return attn_launch(at, c.s);
      });
    }
    B.drop(qk);
    B.drop(vt);
    emit_linear(B, ops, a, nullptr, B.W16(b + ".attn1.o.w"), B.W32(b + ".attn1.o.b"), C, h, &h);
    B.drop(a);
    // cross-attention
    Ten qc = B.alloc(HW, C);
    emit_ln(".ln2", t);
    emit_linear(B, ops, t, nullptr, B.W16(b + ".attn2.q.w"), nullptr, C, qc, nullptr, false,
                fold_of(b + ".attn2.q.wln", b + ".attn2.q"));
    B.drop(t);
    // context K|V of this block: computed once per call into a region reserved
    // before any per-step buffer, so no step op can overwrite it
    const size_t kvoff = kv_regions.at(b);
    const int Lp = (Lc + 7) / 8 * 8;
    const size_t vtoff = kvoff + align_up((size_t)B.Rmax_ * Lc * C * 2, 256);
    a = B.alloc(HW, C);
    {
      const size_t qo = qc.off, ao = a.off;
      const int64_t vld = (int64_t)B.Rmax_ * Lp;
      ops.push_back([=](const RunCtx& c) {
        AttnArgs at{};
        at.q = H16(c, qo);
        at.k = H16(c, kvoff);
        at.vt = H16(c, vtoff);
        at.o = H16(c, ao);
        at.ldq = C;
        at.ldk = C;
        at.ldo = C;
        at.vt_ld = vld;
        at.vt_row = Lp;
        at.rows = c.R;
        at.S = HW;
        at.L = Lc;
        at.heads = heads;
        at.dh = dh;
        at.scale = scale;
        return attn_launch(at, c.s);
      });
    }
    B.drop(qc);
    emit_linear(B, ops, a, nullptr, B.W16(b + ".attn2.o.w"), B.W32(b + ".attn2.o.b"), C, h, &h);
    B.drop(a);
    // GEGLU feed-forward
    Ten f = B.alloc(HW, 4 * C);
    emit_ln(".ln3", t);
    emit_linear(B, ops, t, nullptr, B.W16(b + ".ff1.w"), B.W32(b + ".ff1.b"), 8 * C, f, nullptr,
                true, fold_of(b + ".ff1.wln", b + ".ff1"));
    B.drop(t);
    emit_linear(B, ops, f, nullptr, B.W16(b + ".ff2.w"), B.W32(b + ".ff2.b"), C, h, &h);
    B.drop(f);
  }
  Ten out = B.alloc(HW, C);
  emit_linear(B, ops, h, nullptr, B.W16(n + ".proj_out.w"), B.W32(n + ".proj_out.b"), C, out, &x);
  B.drop(h);
  return out;
}

std::unique_ptr<Plan> build_plan(nv_unet* net, int Rmax) {
  auto P = std::make_unique<Plan>();
  P->Rmax = Rmax;
  const auto& c = net->cfg;
  Builder B(net, P.get(), Rmax);
  const int Bs = (Rmax + 1) / 2;
  const int HW0 = c.H * c.W, C0 = c.ch[0], td = 4 * C0, L = c.n_levels;
  // fixed regions
  P->x_work = B.fixed((size_t)Bs * c.in_ch * HW0 * 4);
  P->eps = B.fixed((size_t)Rmax * HW0 * c.out_ch * 4);
  P->ts = B.fixed(1024 * 4);
  P->at = B.fixed(1024 * 4);
  P->ap = B.fixed(1024 * 4);
  P->ctx = B.fixed((size_t)Rmax * c.ctx_len * c.ctx_dim * 2);
  P->pooled = B.fixed((size_t)Bs * std::max(c.pooled_dim, 1) * 4);
  P->tproj = B.fixed((size_t)Rmax * net->temb_total * 4);
  int maxG = c.gn_groups;
  P->gnpart = B.fixed((size_t)Rmax * ceil_div(HW0, 8) * maxG * 2 * 4);
  P->splitk = B.fixed(SPLITK_BYTES);
  P->stepdev = B.fixed((size_t)2 * MAX_SAMPLES * 4);
  // per-call context K|V regions, one per transformer block
  std::map<std::string, size_t> kv_regions;
  std::map<std::string, int> kv_width;
  for (auto& p : net->params) {
    const std::string& n = p.name;
    const std::string suf = ".attn2.k.w";
    if (n.size() > suf.size() && n.compare(n.size() - suf.size(), suf.size(), suf) == 0) {
      const std::string b = n.substr(0, n.size() - suf.size());
      kv_width[b] = (int)p.shape[0];
      // K rows [Rmax * Lc][C], then V^T [C][Rmax * Lp] (Lp = Lc rounded up to 8)
      const size_t Lp = (c.ctx_len + 7) / 8 * 8;
      kv_regions[b] = B.fixed(align_up((size_t)Rmax * c.ctx_len * p.shape[0] * 2, 256) +
                              (size_t)p.shape[0] * Rmax * Lp * 2);
    }
  }
  auto& ops = P->step;

  // time embedding -> SiLU(temb) -> every ResBlock's projection.  Without a
  // pooled vector the projections depend only on the grid step, so each call
  // computes them once for its N grid steps (P->ttab) and a step copies the
  // rows of its samples' grid steps; with one, every step computes them for
  // its rows.
  if (c.pooled_dim == 0 && net->temb_total % 4 == 0) {
    const int N = net->temb_total;
    P->ttab = B.fixed((size_t)MAX_GRID_STEPS * N * 4);
    const size_t so = B.fixed((size_t)MAX_GRID_STEPS * C0 * 2);
    const size_t o1 = B.fixed((size_t)MAX_GRID_STEPS * td * 2);
    const size_t o2 = B.fixed((size_t)MAX_GRID_STEPS * td * 2);
    const size_t tso = P->ts, tt = P->ttab;
    const _Float16* w1 = B.W16("time.l1.w");
    const float* b1 = B.W32("time.l1.b");
    const _Float16* w2 = B.W16("time.l2.w");
    const float* b2 = B.W32("time.l2.b");
    const _Float16* wa = B.W16("temb_all.w");
    const float* ba = B.W32("temb_all.b");
    P->pre.push_back([=](const RunCtx& x) {
      const int M = x.nsteps;
      if (M < 1 || M > MAX_GRID_STEPS) return hipErrorInvalidValue;
      hipError_t e = temb_sin_steps_launch((const int32_t*)(x.ws + tso), C0, M,
                                           (_Float16*)(x.ws + so), x.s);
      if (e != hipSuccess) return e;
      GemmArgs g = dense_args(td, C0, w1, b1);
      g.M = M;
      g.src1 = (const _Float16*)(x.ws + so);
      g.silu = 1;
      g.out = x.ws + o1;
      g.ldo = td;
      if ((e = gemm_run(g, x)) != hipSuccess) return e;
      g = dense_args(td, td, w2, b2);
      g.M = M;
      g.src1 = (const _Float16*)(x.ws + o1);
      g.silu = 1;
      g.out = x.ws + o2;
      g.ldo = td;
      if ((e = gemm_run(g, x)) != hipSuccess) return e;
      g = dense_args(N, td, wa, ba);
      g.M = M;
      g.src1 = (const _Float16*)(x.ws + o2);
      g.out = x.ws + tt;
      g.ldo = N;
      g.out_f32 = 1;
      return gemm_run(g, x);
    });
    const size_t o = P->tproj;
    ops.push_back([=](const RunCtx& x) {
      return step_rows_launch(x.st, (const float*)(x.ws + tt), N, x.R, (float*)(x.ws + o), x.s);
    });
  } else {
    Ten s0 = B.alloc(1, C0);
    const size_t so = s0.off, tso = P->ts;
    ops.push_back([=](const RunCtx& x) {
      return temb_sin_launch(x.st, (const int32_t*)(x.ws + tso), C0, x.R, H16(x, so), x.s);
    });
    Ten t1 = B.alloc(1, td);
    {
      const _Float16* w = B.W16("time.l1.w");
      const float* b = B.W32("time.l1.b");
      const size_t o = t1.off;
      ops.push_back([=](const RunCtx& x) {
        GemmArgs g = dense_args(td, C0, w, b);
        g.M = x.R;
        g.src1 = H16(x, so);
        g.silu = 1;
        g.out = x.ws + o;
        g.ldo = td;
        return gemm_run(g, x);
      });
    }
    B.drop(s0);
    Ten t2 = B.alloc(1, td);
    {
      const _Float16* w = B.W16("time.l2.w");
      const float* b = B.W32("time.l2.b");
      const size_t i1 = t1.off, o = t2.off, po = P->pooled;
      const bool pooled = c.pooled_dim > 0;
      ops.push_back([=](const RunCtx& x) {
        GemmArgs g = dense_args(td, td, w, b);
        g.M = x.R;
        g.src1 = H16(x, i1);
        if (pooled) {
          g.rowvec = F32(x, po);
          g.rows_div = 2;
          g.ld_rowvec = td;
        }
        g.silu = 1;
        g.out = x.ws + o;
        g.ldo = td;
        return gemm_run(g, x);
      });
    }
    B.drop(t1);
    {
      const _Float16* w = B.W16("temb_all.w");
      const float* b = B.W32("temb_all.b");
      const size_t i2 = t2.off, o = P->tproj;
      const int N = net->temb_total;
      ops.push_back([=](const RunCtx& x) {
        GemmArgs g = dense_args(N, td, w, b);
        g.M = x.R;
        g.src1 = H16(x, i2);
        g.out = x.ws + o;
        g.ldo = N;
        g.out_f32 = 1;
        return gemm_run(g, x);
      });
    }
    B.drop(t2);
  }
  // conv_in on the float32 latent
  Ten h = B.alloc(HW0, C0);
  {
    const float* w = B.W32("conv_in.w");
    const float* b = B.W32("conv_in.b");
    const size_t o = h.off;
    const int cin = c.in_ch, H = c.H, W = c.W;
    ops.push_back([=](const RunCtx& x) {
      return conv_in_launch(x.x, w, b, cin, H, W, C0, x.R, H16(x, o), x.s);
    });
  }
  std::vector<Ten> skips;
  skips.push_back(h);
  B.hold(h);
  int H = c.H, W = c.W;
  for (int lv = 0; lv < L; ++lv) {
    const int co = c.ch[lv];
    for (int r = 0; r < c.n_res; ++r) {
      const std::string base = "down" + std::to_string(lv);
      Ten nh = build_res(B, ops, h, nullptr, base + ".res" + std::to_string(r), co, H, W);
      B.drop(h);
      h = nh;
      if (c.depth[lv] > 0) {
        nh = build_tr(B, ops, h, base + ".attn" + std::to_string(r), c.depth[lv], H, W,
                      kv_regions);
        B.drop(h);
        h = nh;
      }
      skips.push_back(h);
      B.hold(h);
    }
    if (lv < L - 1) {
      Ten nh = B.alloc((H / 2) * (W / 2), h.C);
      emit_conv(B, ops, h, nullptr, "down" + std::to_string(lv) + ".ds", h.C,
                {H, W, H / 2, W / 2, 2, 0}, nh, nullptr, -1);
      B.drop(h);
      h = nh;
      H /= 2;
      W /= 2;
      skips.push_back(h);
      B.hold(h);
    }
  }
  {
    Ten nh = build_res(B, ops, h, nullptr, "mid.res0", h.C, H, W);
    B.drop(h);
    h = nh;
    if (c.mid_depth > 0) {
      nh = build_tr(B, ops, h, "mid.attn", c.mid_depth, H, W, kv_regions);
      B.drop(h);
      h = nh;
    }
    nh = build_res(B, ops, h, nullptr, "mid.res1", h.C, H, W);
    B.drop(h);
    h = nh;
  }
  for (int lv = L - 1; lv >= 0; --lv) {
    const int co = c.ch[lv];
    const std::string base = "up" + std::to_string(lv);
    for (int r = 0; r < c.n_res + 1; ++r) {
      Ten sk = skips.back();
      skips.pop_back();
      Ten nh = build_res(B, ops, h, &sk, base + ".res" + std::to_string(r), co, H, W);
      B.drop(h);
      B.drop(sk);
      h = nh;
      if (c.depth[lv] > 0) {
        nh = build_tr(B, ops, h, base + ".attn" + std::to_string(r), c.depth[lv], H, W,
                      kv_regions);
        B.drop(h);
        h = nh;
      }
    }
    if (lv > 0) {
      Ten nh = B.alloc(4 * H * W, h.C);
      emit_conv(B, ops, h, nullptr, base + ".us", h.C, {H, W, 2 * H, 2 * W, 1, 1}, nh, nullptr,
                -1);
      B.drop(h);
      h = nh;
      H *= 2;
      W *= 2;
    }
  }
  {
    Ten a = B.alloc(HW0, h.C);
    emit_gn(B, ops, h, nullptr, "out.gn", true, a);
    B.drop(h);
    emit_conv(B, ops, a, nullptr, "conv_out", c.out_ch, {H, W, H, W, 1, 0}, a, nullptr, -1, true,
              P->eps);
    B.drop(a);
  }
  // per-call context projections
  for (auto& kr : kv_regions) {
    const std::string b = kr.first;
    const size_t kvoff = kr.second, ctxo = P->ctx;
    const _Float16* w = B.W16(b + ".attn2.kv.w");
    const int Lc = c.ctx_len, D = c.ctx_dim;
    const int C = kv_width.at(b);
    const int Lp = (Lc + 7) / 8 * 8;
    const size_t vtoff = kvoff + align_up((size_t)Rmax * Lc * C * 2, 256);
    P->pre.push_back([=](const RunCtx& x) {
      GemmArgs g = dense_args(2 * C, D, w, nullptr);
      g.M = (int64_t)x.R * Lc;
      g.src1 = H16(x, ctxo);
      g.out = x.ws + kvoff;
      g.ldo = C;
      g.vt = H16(x, vtoff);
      g.vt_col0 = C;
      g.vt_ld = (int64_t)Rmax * Lp;
      g.vt_div = Lc;
      g.vt_stride = Lp;
      return gemm_run(g, x);
    });
  }
  P->bytes = align_up(B.peak(), 256);
  return P;
}

Plan* get_plan(nv_unet* net, int Rmax) {
  auto it = net->plans.find(Rmax);
  if (it != net->plans.end()) return it->second.get();
  auto p = build_plan(net, Rmax);
  Plan* raw = p.get();
  net->plans[Rmax] = std::move(p);
  return raw;
}

// Host-side weight packing ------------------------------------------------
bool pack_weights(nv_unet* net, const float* blob) {
  const auto& c = net->cfg;
  std::map<std::string, const ParamInfo*> by;
  for (auto& p : net->params) by[p.name] = &p;
  auto P = [&](const std::string& n) -> const float* { return blob + by.at(n)->offset; };
  auto S = [&](const std::string& n) -> const std::vector<int64_t>& { return by.at(n)->shape; };
  std::vector<_Float16> h16;
  std::vector<float> h32;
  std::map<std::string, size_t> o16, o32;
  auto put32 = [&](const std::string& n, const float* src, int64_t cnt) {
    o32[n] = h32.size();
    h32.insert(h32.end(), src, src + cnt);
    while (h32.size() % 64) h32.push_back(0.f);
  };
  auto begin16 = [&](const std::string& n) { o16[n] = h16.size(); };
  auto end16 = [&]() {
    while (h16.size() % 128) h16.push_back((_Float16)0.f);
  };
  // One weight row W[n][0..K) to float16; with a folded LayerNorm (gam, bet
  // non-null) the row is gamma-scaled and c1 / c2 gain
  // sum_k float16(gamma_k W[n][k]) and bias + sum_k beta_k W[n][k] (float64 sums).
  auto push_row = [&](const float* wr, int K, const float* gam, const float* bet, double bias,
                      std::vector<float>& c1, std::vector<float>& c2) {
    if (!gam) {
      for (int k = 0; k < K; ++k) h16.push_back((_Float16)wr[k]);
      return;
    }
    double s1 = 0.0, s2 = bias;
    for (int k = 0; k < K; ++k) {
      const _Float16 h = (_Float16)(gam[k] * wr[k]);
      h16.push_back(h);
      s1 += (double)(float)h;
      s2 += (double)bet[k] * (double)wr[k];
    }
    c1.push_back((float)s1);
    c2.push_back((float)s2);
  };
  // ResBlock time projections stacked
  int ttot = 0;
  for (auto& p : net->params) {
    const std::string& n = p.name;
    if (n.size() > 7 && n.compare(n.size() - 7, 7, ".temb.w") == 0) {
      net->temb_off[n.substr(0, n.size() - 7)] = ttot;
      ttot += (int)p.shape[0];
    }
  }
  net->temb_total = ttot;
  {
    begin16("temb_all.w");
    std::vector<float> bias;
    for (auto& p : net->params) {
      const std::string& n = p.name;
      if (n.size() > 7 && n.compare(n.size() - 7, 7, ".temb.w") == 0) {
        const float* src = blob + p.offset;
        for (int64_t i = 0; i < p.numel(); ++i) h16.push_back((_Float16)src[i]);
        const std::string bn = n.substr(0, n.size() - 1) + "b";
        const float* bs = P(bn);
        bias.insert(bias.end(), bs, bs + p.shape[0]);
      }
    }
    end16();
    put32("temb_all.b", bias.data(), (int64_t)bias.size());
  }
  for (auto& p : net->params) {
    const std::string& n = p.name;
    const float* src = blob + p.offset;
    auto ends = [&](const char* suf) {
      const size_t l = strlen(suf);
      return n.size() >= l && n.compare(n.size() - l, l, suf) == 0;
    };
    if (ends(".temb.w") || ends(".temb.b")) continue;
    if (n == "conv_in.w") {
      put32(n, src, p.numel());
      continue;
    }
    if (p.shape.size() == 1) {
      if (ends(".ff1.b")) {  // GEGLU packing of the bias
        const int C8 = (int)p.shape[0], C4 = C8 / 2;
        std::vector<float> pk(C8);
        for (int r = 0; r < C8; ++r) {
          const int grp = r / 32, wi = r % 32;
          pk[r] = wi < 16 ? src[grp * 16 + wi] : src[C4 + grp * 16 + (wi - 16)];
        }
        put32(n, pk.data(), C8);
      } else {
        put32(n, src, p.numel());
      }
      continue;
    }
    if (p.shape.size() == 4) {  // [Co][Ci][3][3] -> [Co][3][3][Ci]
      const int co = (int)p.shape[0], ci = (int)p.shape[1];
      begin16(n);
      for (int o = 0; o < co; ++o)
        for (int t = 0; t < 9; ++t)
          for (int i = 0; i < ci; ++i) h16.push_back((_Float16)src[((int64_t)o * ci + i) * 9 + t]);
      end16();
      continue;
    }
    // 2-D linear weights
    if (ends(".attn1.q.w")) {
      const std::string b = n.substr(0, n.size() - 10);  // strip ".attn1.q.w"
      const int K = (int)p.shape[1];
      std::vector<float> c1, c2;
      for (const bool fold : {false, true}) {
        if (fold && !ln_folded(K)) break;
        const float* gam = fold ? P(b + ".ln1.g") : nullptr;
        const float* bet = fold ? P(b + ".ln1.b") : nullptr;
        begin16(b + (fold ? ".attn1.qkv.wln" : ".attn1.qkv.w"));
        for (const char* part : {".attn1.q.w", ".attn1.k.w", ".attn1.v.w"}) {
          const float* s2 = P(b + part);
          for (int64_t r = 0; r < S(b + part)[0]; ++r)
            push_row(s2 + r * K, K, gam, bet, 0.0, c1, c2);
        }
        end16();
      }
      if (!c1.empty()) {
        put32(b + ".attn1.qkv.c1", c1.data(), (int64_t)c1.size());
        put32(b + ".attn1.qkv.c2", c2.data(), (int64_t)c2.size());
      }
      continue;
    }
    if (ends(".attn2.q.w") && ln_folded((int)p.shape[1])) {
      const std::string b = n.substr(0, n.size() - 10);  // strip ".attn2.q.w"
      const int K = (int)p.shape[1];
      std::vector<float> c1, c2;
      for (const bool fold : {false, true}) {
        begin16(fold ? b + ".attn2.q.wln" : n);
        for (int64_t r = 0; r < p.shape[0]; ++r)
          push_row(src + r * K, K, fold ? P(b + ".ln2.g") : nullptr,
                   fold ? P(b + ".ln2.b") : nullptr, 0.0, c1, c2);
        end16();
      }
      put32(b + ".attn2.q.c1", c1.data(), (int64_t)c1.size());
      put32(b + ".attn2.q.c2", c2.data(), (int64_t)c2.size());
      continue;
    }
    if (ends(".attn1.k.w") || ends(".attn1.v.w") || ends(".attn2.v.w")) continue;
    if (ends(".attn2.k.w")) {
      const std::string b = n.substr(0, n.size() - 10);
      begin16(b + ".attn2.kv.w");
      for (const char* part : {".attn2.k.w", ".attn2.v.w"}) {
        const float* s2 = P(b + part);
        const int64_t cnt = S(b + part)[0] * S(b + part)[1];
        for (int64_t i = 0; i < cnt; ++i) h16.push_back((_Float16)s2[i]);
      }
      end16();
      continue;
    }
    if (ends(".ff1.w")) {
      const std::string b = n.substr(0, n.size() - 6);  // strip ".ff1.w"
      const int C8 = (int)p.shape[0], C4 = C8 / 2, K = (int)p.shape[1];
      const float* bias = P(b + ".ff1.b");
      std::vector<float> c1, c2;
      for (const bool fold : {false, true}) {
        if (fold && !ln_folded(K)) break;
        const float* gam = fold ? P(b + ".ln3.g") : nullptr;
        const float* bet = fold ? P(b + ".ln3.b") : nullptr;
        begin16(fold ? b + ".ff1.wln" : n);
        for (int r = 0; r < C8; ++r) {
          const int grp = r / 32, wi = r % 32;
          const int srow = wi < 16 ? grp * 16 + wi : C4 + grp * 16 + (wi - 16);
          push_row(src + (int64_t)srow * K, K, gam, bet, bias[srow], c1, c2);
        }
        end16();
      }
      if (!c1.empty()) {
        put32(b + ".ff1.c1", c1.data(), (int64_t)c1.size());
        put32(b + ".ff1.c2", c2.data(), (int64_t)c2.size());
      }
      continue;
    }
    begin16(n);
    for (int64_t i = 0; i < p.numel(); ++i) h16.push_back((_Float16)src[i]);
    end16();
  }
  if (hipMalloc((void**)&net->d16, std::max<size_t>(h16.size(), 1) * 2) != hipSuccess) return false;
  if (hipMalloc((void**)&net->d32, std::max<size_t>(h32.size(), 1) * 4) != hipSuccess) return false;
  if (hipMemcpy(net->d16, h16.data(), h16.size() * 2, hipMemcpyHostToDevice) != hipSuccess)
    return false;
  if (hipMemcpy(net->d32, h32.data(), h32.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
    return false;
  for (auto& kv : o16) net->w16[kv.first] = net->d16 + kv.second;
  for (auto& kv : o32) net->w32[kv.first] = net->d32 + kv.second;
  (void)c;
  return true;
}

int32_t check_sched(const nv_schedule* s) {
  NV_CHECK_ARG(s, "null schedule");
  NV_CHECK_ARG(s->N >= 1 && s->T >= 2 && s->T <= 1024, "need 1 <= N, 2 <= T <= 1024");
  NV_CHECK_ARG(s->T % s->N == 0 && s->T / s->N >= 2, "T must be a multiple of N with T/N >= 2");
  NV_CHECK_ARG(s->beta_start > 0 && s->beta_end > 0 && s->beta_start < 1 && s->beta_end < 1,
               "betas must be in (0, 1)");
  return NV_OK;
}

hipError_t run_ops(const std::vector<Op>& ops, const RunCtx& c) {
  for (const auto& op : ops) {
    hipError_t e = op(c);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace
}  // namespace nv

using namespace nv;

extern "C" const char* nv_status_string(int32_t s) {
  switch (s) {
    case NV_OK: return "ok";
    case NV_ERR_INVALID_ARG: return "invalid argument";
    case NV_ERR_UNSUPPORTED: return "unsupported";
    case NV_ERR_OUT_OF_MEMORY: return "out of device memory";
    case NV_ERR_HIP: return "HIP runtime error";
    case NV_ERR_WORKSPACE: return "workspace missing or too small";
    default: return "unknown status";
  }
}

extern "C" const char* nv_last_error(void) { return g_err.c_str(); }
extern "C" const char* nv_version(void) { return "nv 0.1 (gfx950)"; }

extern "C" int64_t nv_unet_param_count(const nv_unet_config* cfg) {
  std::string why;
  if (!validate_cfg(cfg, &why)) {
    set_error(why);
    return -1;
  }
  std::vector<ParamInfo> ps;
  enumerate_params(*cfg, ps);
  int64_t n = 0;
  for (auto& p : ps) n += p.numel();
  return n;
}

extern "C" int32_t nv_unet_param_info(const nv_unet_config* cfg, int64_t i, char* name,
                                      int32_t name_len, int64_t* numel) {
  std::string why;
  if (!validate_cfg(cfg, &why)) {
    set_error(why);
    return NV_ERR_INVALID_ARG;
  }
  std::vector<ParamInfo> ps;
  enumerate_params(*cfg, ps);
  NV_CHECK_ARG(i >= 0 && i < (int64_t)ps.size(), "parameter index out of range");
  NV_CHECK_ARG(name && name_len > 0, "null name buffer");
  snprintf(name, (size_t)name_len, "%s", ps[i].name.c_str());
  if (numel) *numel = ps[i].numel();
  return NV_OK;
}

extern "C" int32_t nv_unet_create(const nv_unet_config* cfg, const float* weights_host,
                                  int64_t n_weights, nv_unet** out) {
  clear_error();
  NV_CHECK_ARG(out && weights_host, "null output or weights pointer");
  std::string why;
  if (!validate_cfg(cfg, &why)) {
    set_error(why);
    return NV_ERR_INVALID_ARG;
  }
  auto net = std::make_unique<nv_unet>();
  net->cfg = *cfg;
  enumerate_params(*cfg, net->params);
  int64_t total = 0;
  for (auto& p : net->params) total += p.numel();
  NV_CHECK_ARG(n_weights == total, "n_weights does not match nv_unet_param_count");
  if (!pack_weights(net.get(), weights_host)) {
    if (net->d16) (void)hipFree(net->d16);
    if (net->d32) (void)hipFree(net->d32);
    set_error("device allocation or copy of the weights failed");
    return NV_ERR_OUT_OF_MEMORY;
  }
  *out = net.release();
  return NV_OK;
}

extern "C" void nv_unet_destroy(nv_unet* net) {
  if (!net) return;
  net->drop_graphs();
  if (net->capture_stream) (void)hipStreamDestroy(net->capture_stream);
  if (net->d16) (void)hipFree(net->d16);
  if (net->d32) (void)hipFree(net->d32);
  delete net;
}

extern "C" size_t nv_denoise_workspace(const nv_unet* cnet, int32_t B) {
  if (!cnet || B < 1 || B > MAX_SAMPLES) return 0;
  nv_unet* net = const_cast<nv_unet*>(cnet);
  try {
    return get_plan(net, 2 * B)->bytes;
  } catch (const std::exception& e) {
    set_error(e.what());
    return 0;
  }
}

namespace {
int32_t prep_call(nv_unet* net, const nv_schedule* sched, int32_t B, const float* cond,
                  const float* uncond, const float* pooled, void* workspace, size_t ws_bytes,
                  Plan** plan) {
  NV_CHECK_ARG(net, "null handle");
  int32_t st = check_sched(sched);
  if (st != NV_OK) return st;
  NV_CHECK_ARG(B >= 1 && B <= MAX_SAMPLES, "B must be in [1, 64]");
  NV_CHECK_ARG(cond && uncond, "null context pointer");
  NV_CHECK_ARG(net->cfg.pooled_dim == 0 || pooled, "pooled vector required by this topology");
  Plan* p = nullptr;
  try {
    p = get_plan(net, 2 * B);
  } catch (const std::exception& e) {
    set_error(e.what());
    return NV_ERR_INVALID_ARG;
  }
  if (!workspace || ws_bytes < p->bytes || ((uintptr_t)workspace & 255)) {
    set_error("denoise workspace missing, misaligned or smaller than nv_denoise_workspace()");
    return NV_ERR_WORKSPACE;
  }
  *plan = p;
  return NV_OK;
}
}  // namespace

// Snapshots of the cache-miss path: the state of sample b after slot_k[s]
// steps goes to state dst[b][s] of store (dst < 0: not stored).
struct Snapshots {
  float* store = nullptr;
  int n_slots = 0;
  int32_t slot_k[16] = {};
  std::vector<int64_t> dst;  // [B][n_slots]
};

// Stochastic DDIM (eta > 0): the caller's standard normal draws per sample and
// grid step, device f32 [B][N][latent].
struct Stochastic {
  float eta = 0.0f;
  const float* z = nullptr;
};

static int32_t denoise_impl(nv_unet* net, const nv_schedule* sched, float* latent,
                            const int32_t* k, int32_t B, const float* cond, const float* uncond,
                            const float* pooled, float guidance, void* workspace,
                            size_t workspace_bytes, void* stream, const Snapshots* snap,
                            const Stochastic* sto = nullptr) {
  NV_CHECK_ARG(latent && k, "null latent or k");
  NV_CHECK_ARG(std::isfinite(guidance), "guidance must be finite");
  Plan* P = nullptr;
  int32_t st = prep_call(net, sched, B, cond, uncond, pooled, workspace, workspace_bytes, &P);
  if (st != NV_OK) return st;
  const int N = sched->N;
  for (int b = 0; b < B; ++b) NV_CHECK_ARG(k[b] >= 0 && k[b] <= N, "k[b] must be in [0, N]");
  const auto& c = net->cfg;
  StepArgs sa{};
  std::vector<int> order(B);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return k[a] < k[b]; });
  for (int b = 0; b < B; ++b) {
    sa.perm[b] = order[b];
    sa.kstep[b] = k[order[b]];
  }
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  sa.dev = (int32_t*)(ws + P->stepdev);
  const int HW = c.H * c.W;
  const int64_t lat = (int64_t)c.in_ch * HW;
  NV_HIP_TRY(schedule_launch(sched->T, N, sched->beta_start, sched->beta_end,
                             (int32_t*)(ws + P->ts), (float*)(ws + P->at), (float*)(ws + P->ap),
                             s));
  NV_HIP_TRY(steps_init_launch(sa, s));
  NV_HIP_TRY(permute_launch(sa, latent, (float*)(ws + P->x_work), lat, B, 1, s));
  NV_HIP_TRY(ctx_rows_launch(sa, cond, uncond, (int64_t)c.ctx_len * c.ctx_dim, 2 * B,
                             (_Float16*)(ws + P->ctx), s));
  if (c.pooled_dim > 0)
    NV_HIP_TRY(permute_launch(sa, pooled, (float*)(ws + P->pooled), c.pooled_dim, B, 1, s));
  RunCtx rc{ws, 2 * B, s, (const float*)(ws + P->x_work), sa, (float*)(ws + P->splitk),
            SPLITK_BYTES};
  rc.nsteps = N;
  // copy every sorted sample a whose step count equals a slot's K
  auto take = [&](int a, int done) -> hipError_t {
    if (!snap) return hipSuccess;
    const int b = sa.perm[a];
    for (int q = 0; q < snap->n_slots; ++q)
      if (snap->slot_k[q] == done && snap->dst[(size_t)b * snap->n_slots + q] >= 0) {
        const int64_t to = snap->dst[(size_t)b * snap->n_slots + q];
        hipError_t err = hipMemcpyAsync(snap->store + to * lat,
                                        (const float*)(ws + P->x_work) + a * lat, lat * 4,
                                        hipMemcpyDeviceToDevice, s);
        if (err != hipSuccess) return err;
      }
    return hipSuccess;
  };
  for (int a = 0; a < B; ++a) NV_HIP_TRY(take(a, sa.kstep[a]));  // the states given
  NV_HIP_TRY(run_ops(P->pre, rc));
  // One step for the first A samples: the UNet on their 2A rows, guidance and
  // the DDIM update, then every sample's grid step moves on.  Enqueued on
  // stream `on`.
  const float eta = sto ? sto->eta : 0.0f;
  const float* z = sto ? sto->z : nullptr;
  auto step_ops = [&](int A, hipStream_t on) -> hipError_t {
    RunCtx r = rc;
    r.R = 2 * A;
    r.s = on;
    hipError_t e = run_ops(P->step, r);
    if (e == hipSuccess)
      e = cfg_ddim_launch(r.st, (const float*)(ws + P->eps), (float*)(ws + P->x_work), c.out_ch,
                          HW, A, guidance, (const float*)(ws + P->at), (const float*)(ws + P->ap),
                          eta, z, N, on);
    if (e == hipSuccess) e = steps_advance_launch(sa.dev, on);
    return e;
  };
  // Replayed from a graph captured on first use (per active row count, for
  // this plan, workspace and update), unless launches are being traced.
  const GraphKey key{P, ws, guidance, eta, z, N};
  const bool graphs = net->use_graphs && !trace_active();
  if (graphs && !(key == net->gkey)) {
    net->drop_graphs();
    net->gkey = key;
  }
  auto graph_for = [&](int A) -> hipGraphExec_t {
    auto it = net->graphs.find(A);
    if (it != net->graphs.end()) return it->second;
    if (!net->capture_stream &&
        hipStreamCreateWithFlags(&net->capture_stream, hipStreamNonBlocking) != hipSuccess)
      return nullptr;
    hipGraph_t g = nullptr;
    hipGraphExec_t ex = nullptr;
    if (hipStreamBeginCapture(net->capture_stream, hipStreamCaptureModeRelaxed) != hipSuccess)
      return nullptr;
    const hipError_t e = step_ops(A, net->capture_stream);
    const hipError_t ee = hipStreamEndCapture(net->capture_stream, &g);
    if (e == hipSuccess && ee == hipSuccess && g &&
        hipGraphInstantiate(&ex, g, nullptr, nullptr, 0) == hipSuccess) {
      net->graphs[A] = ex;
    } else {
      ex = nullptr;
    }
    if (g) (void)hipGraphDestroy(g);
    (void)hipGetLastError();  // a failed capture leaves no sticky error behind
    return ex;
  };
  for (int j = 0;; ++j) {
    int A = 0;
    while (A < B && sa.kstep[A] + j < N) ++A;
    if (A == 0) break;
    hipGraphExec_t ex = graphs && net->use_graphs ? graph_for(A) : nullptr;
    if (ex) {
      NV_HIP_TRY(hipGraphLaunch(ex, s));
    } else {
      if (graphs) net->use_graphs = false;  // capture failed: launch eagerly from now on
      NV_HIP_TRY(step_ops(A, s));
    }
    for (int a = 0; a < A; ++a) NV_HIP_TRY(take(a, sa.kstep[a] + j + 1));
  }
  NV_HIP_TRY(permute_launch(sa, (const float*)(ws + P->x_work), latent, lat, B, 0, s));
  return NV_OK;
}

extern "C" int32_t nv_denoise(nv_unet* net, const nv_schedule* sched, float* latent,
                              const int32_t* k, int32_t B, const float* cond,
                              const float* uncond, const float* pooled, float guidance,
                              void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  return denoise_impl(net, sched, latent, k, B, cond, uncond, pooled, guidance, workspace,
                      workspace_bytes, stream, nullptr);
}

extern "C" int32_t nv_denoise_eta(nv_unet* net, const nv_schedule* sched, float* latent,
                                  const int32_t* k, int32_t B, const float* cond,
                                  const float* uncond, const float* pooled, float guidance,
                                  float eta, const float* noise, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  clear_error();
  NV_CHECK_ARG(noise, "null noise");
  NV_CHECK_ARG(eta >= 0.0f && eta <= 1.0f, "eta must be in [0, 1]");
  Stochastic sto;
  sto.eta = eta;
  sto.z = noise;
  return denoise_impl(net, sched, latent, k, B, cond, uncond, pooled, guidance, workspace,
                      workspace_bytes, stream, nullptr, &sto);
}

extern "C" int32_t nv_denoise_store(nv_unet* net, const nv_schedule* sched, float* latent,
                                    const int32_t* k, int32_t B, const float* cond,
                                    const float* uncond, const float* pooled, float guidance,
                                    float* store, int64_t n_store, int32_t n_slots,
                                    const int32_t* slot_k, const int64_t* entry,
                                    void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  NV_CHECK_ARG(n_slots >= 1 && n_slots <= 16 && slot_k && entry, "need 1..16 slots and entries");
  NV_CHECK_ARG(sched, "null schedule");
  NV_CHECK_ARG(B >= 1 && B <= MAX_SAMPLES, "B must be in [1, 64]");
  Snapshots sn;
  sn.store = store;
  sn.n_slots = n_slots;
  for (int q = 0; q < n_slots; ++q) {
    NV_CHECK_ARG(slot_k[q] >= 0 && slot_k[q] <= sched->N, "slot_k must be in [0, N]");
    sn.slot_k[q] = slot_k[q];
  }
  bool any = false;
  sn.dst.assign((size_t)B * n_slots, -1);
  for (int b = 0; b < B; ++b) {
    NV_CHECK_ARG(entry[b] >= -1 && entry[b] < n_store, "entry[b] must be -1 or in [0, n_store)");
    any |= entry[b] >= 0;
    if (entry[b] >= 0)
      for (int q = 0; q < n_slots; ++q) sn.dst[(size_t)b * n_slots + q] = entry[b] * n_slots + q;
  }
  NV_CHECK_ARG(!any || store, "null store with entries to write");
  return denoise_impl(net, sched, latent, k, B, cond, uncond, pooled, guidance, workspace,
                      workspace_bytes, stream, &sn);
}

extern "C" int32_t nv_denoise_store_pool(nv_unet* net, const nv_schedule* sched, float* latent,
                                         const int32_t* k, int32_t B, const float* cond,
                                         const float* uncond, const float* pooled,
                                         float guidance, float* pool, int64_t n_pool,
                                         int32_t n_slots, const int32_t* slot_k,
                                         const int32_t* dst, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  clear_error();
  NV_CHECK_ARG(n_slots >= 1 && n_slots <= 16 && slot_k && dst, "need 1..16 slots and dst");
  NV_CHECK_ARG(sched, "null schedule");
  NV_CHECK_ARG(B >= 1 && B <= MAX_SAMPLES, "B must be in [1, 64]");
  Snapshots sn;
  sn.store = pool;
  sn.n_slots = n_slots;
  for (int q = 0; q < n_slots; ++q) {
    NV_CHECK_ARG(slot_k[q] >= 0 && slot_k[q] <= sched->N, "slot_k must be in [0, N]");
    sn.slot_k[q] = slot_k[q];
  }
  bool any = false;
  sn.dst.assign((size_t)B * n_slots, -1);
  for (int64_t i = 0; i < (int64_t)B * n_slots; ++i) {
    NV_CHECK_ARG(dst[i] >= -1 && dst[i] < n_pool, "dst must be -1 or in [0, n_pool)");
    any |= dst[i] >= 0;
    sn.dst[i] = dst[i];
  }
  NV_CHECK_ARG(!any || pool, "null pool with states to write");
  // two writes to one state would leave whichever ran last
  std::vector<int32_t> used;
  for (int64_t i = 0; i < (int64_t)B * n_slots; ++i)
    if (dst[i] >= 0) used.push_back(dst[i]);
  std::sort(used.begin(), used.end());
  NV_CHECK_ARG(std::adjacent_find(used.begin(), used.end()) == used.end(),
               "dst names one state twice");
  return denoise_impl(net, sched, latent, k, B, cond, uncond, pooled, guidance, workspace,
                      workspace_bytes, stream, &sn);
}

extern "C" int32_t nv_unet_eps(nv_unet* net, const nv_schedule* sched, const float* x,
                               const int32_t* step_idx, int32_t B, const float* cond,
                               const float* uncond, const float* pooled, float* eps_uncond,
                               float* eps_cond, void* workspace, size_t workspace_bytes,
                               void* stream) {
  clear_error();
  NV_CHECK_ARG(x && step_idx && eps_uncond && eps_cond, "null pointer argument");
  Plan* P = nullptr;
  int32_t st = prep_call(net, sched, B, cond, uncond, pooled, workspace, workspace_bytes, &P);
  if (st != NV_OK) return st;
  for (int b = 0; b < B; ++b)
    NV_CHECK_ARG(step_idx[b] >= 0 && step_idx[b] < sched->N, "step_idx must be in [0, N)");
  const auto& c = net->cfg;
  StepArgs sa{};
  for (int b = 0; b < B; ++b) {
    sa.perm[b] = b;
    sa.kstep[b] = step_idx[b];
  }
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  sa.dev = (int32_t*)(ws + P->stepdev);
  NV_HIP_TRY(schedule_launch(sched->T, sched->N, sched->beta_start, sched->beta_end,
                             (int32_t*)(ws + P->ts), (float*)(ws + P->at), (float*)(ws + P->ap),
                             s));
  NV_HIP_TRY(steps_init_launch(sa, s));
  NV_HIP_TRY(ctx_rows_launch(sa, cond, uncond, (int64_t)c.ctx_len * c.ctx_dim, 2 * B,
                             (_Float16*)(ws + P->ctx), s));
  if (c.pooled_dim > 0)
    NV_HIP_TRY(permute_launch(sa, pooled, (float*)(ws + P->pooled), c.pooled_dim, B, 1, s));
  RunCtx rc{ws, 2 * B, s, x, sa, (float*)(ws + P->splitk), SPLITK_BYTES};
  rc.nsteps = sched->N;
  NV_HIP_TRY(run_ops(P->pre, rc));
  NV_HIP_TRY(run_ops(P->step, rc));
  NV_HIP_TRY(eps_split_launch((const float*)(ws + P->eps), c.out_ch, c.H * c.W, B, eps_uncond,
                              eps_cond, s));
  return NV_OK;
}

extern "C" int32_t nv_unet_set_options(nv_unet* net, int32_t flags) {
  clear_error();
  NV_CHECK_ARG(net, "null handle");
  NV_CHECK_ARG((flags & ~NV_UNET_GRAPHS) == 0, "unknown option flags");
  net->use_graphs = (flags & NV_UNET_GRAPHS) != 0;
  net->drop_graphs();
  net->gkey = GraphKey{};
  return NV_OK;
}

extern "C" size_t nv_op_workspace(void) { return SPLITK_BYTES; }

extern "C" int32_t nv_op_linear(const void* x, const void* x2, const void* w, const float* bias,
                                const void* residual, void* out, int64_t M, int32_t N, int32_t K1,
                                int32_t K2, void* workspace, size_t workspace_bytes,
                                void* stream) {
  clear_error();
  NV_CHECK_ARG(x && w && out, "null pointer argument");
  NV_CHECK_ARG(M >= 1 && N >= 1 && K1 >= 8 && K1 % 8 == 0 && K2 >= 0 && K2 % 8 == 0,
               "need M, N >= 1, K1 >= 8 and K1, K2 multiples of 8");
  NV_CHECK_ARG((K2 == 0) == (x2 == nullptr), "x2 must be given exactly when K2 > 0");
  if (!workspace || workspace_bytes < SPLITK_BYTES || ((uintptr_t)workspace & 255)) {
    set_error("op workspace missing, misaligned or smaller than nv_op_workspace()");
    return NV_ERR_WORKSPACE;
  }
  GemmArgs g = dense_args(N, K1 + K2, (const _Float16*)w, bias);
  g.M = M;
  g.src1 = (const _Float16*)x;
  g.C1 = K1;
  g.lda1 = K1;
  if (x2) {
    g.src2 = (const _Float16*)x2;
    g.C2 = K2;
    g.lda2 = K2;
  }
  if (residual) {
    g.residual = (const _Float16*)residual;
    g.ld_res = N;
  }
  g.out = out;
  g.ldo = N;
  g.partial = (float*)workspace;
  g.partial_bytes = workspace_bytes;
  NV_HIP_TRY(gemm_launch(g, (hipStream_t)stream));
  return NV_OK;
}

extern "C" int32_t nv_op_conv3x3(const void* x, const void* x2, const void* w, const float* bias,
                                 void* out, int32_t B, int32_t H, int32_t W, int32_t Cin1,
                                 int32_t Cin2, int32_t Cout, int32_t stride, int32_t upsample,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  NV_CHECK_ARG(x && w && out, "null pointer argument");
  NV_CHECK_ARG(B >= 1 && H >= 1 && W >= 1 && Cout >= 1 && Cin1 >= 8 && Cin1 % 8 == 0 &&
                   Cin2 >= 0 && Cin2 % 8 == 0,
               "bad conv shape (Cin1, Cin2 multiples of 8)");
  NV_CHECK_ARG((Cin2 == 0) == (x2 == nullptr), "x2 must be given exactly when Cin2 > 0");
  NV_CHECK_ARG(stride == 1 || (stride == 2 && H % 2 == 0 && W % 2 == 0 && !upsample),
               "stride must be 1, or 2 with even H, W and no upsample");
  if (!workspace || workspace_bytes < SPLITK_BYTES || ((uintptr_t)workspace & 255)) {
    set_error("op workspace missing, misaligned or smaller than nv_op_workspace()");
    return NV_ERR_WORKSPACE;
  }
  const int Ho = upsample ? 2 * H : H / stride, Wo = upsample ? 2 * W : W / stride;
  GemmArgs g{};
  g.M = (int64_t)B * Ho * Wo;
  g.N = Cout;
  g.K = 9 * (Cin1 + Cin2);
  g.src1 = (const _Float16*)x;
  g.C1 = Cin1;
  g.src2 = (const _Float16*)x2;
  g.C2 = Cin2;
  g.conv = 1;
  g.Hin = H;
  g.Win = W;
  g.Ho = Ho;
  g.Wo = Wo;
  g.stride = stride;
  g.upsample = upsample ? 1 : 0;
  g.w = (const _Float16*)w;
  g.ldw = g.K;
  g.bias = bias;
  g.rows_div = 1;
  g.out = out;
  g.ldo = Cout;
  g.partial = (float*)workspace;
  g.partial_bytes = workspace_bytes;
  NV_HIP_TRY(gemm_launch(g, (hipStream_t)stream));
  return NV_OK;
}

extern "C" int32_t nv_op_attention(const void* q, const void* k, const void* vt, void* out,
                                   int32_t rows, int32_t S, int32_t L, int32_t heads, int32_t dh,
                                   int32_t ldq, int32_t ldk, int32_t ldo, int64_t vt_ld,
                                   int64_t vt_row, float scale, void* stream) {
  clear_error();
  NV_CHECK_ARG(q && k && vt && out, "null pointer argument");
  NV_CHECK_ARG(rows >= 1 && S >= 1 && L >= 1 && heads >= 1, "sizes must be >= 1");
  NV_CHECK_ARG(ldq >= heads * dh && ldk >= heads * dh && ldo >= heads * dh,
               "row strides smaller than heads * dh");
  NV_CHECK_ARG(ldq % 8 == 0 && ldk % 8 == 0 && ldo % 8 == 0, "row strides must be multiples of 8");
  NV_CHECK_ARG(vt_row >= L && vt_row % 8 == 0 && vt_ld % 8 == 0 && vt_ld >= rows * vt_row,
               "bad transposed-V layout");
  NV_CHECK_ARG(std::isfinite(scale), "scale must be finite");
  if (!attn_supported(dh)) {
    set_error("head dim must be one of 16, 32, 40, 64, 80, 128, 160");
    return NV_ERR_UNSUPPORTED;
  }
  AttnArgs a{};
  a.q = (const _Float16*)q;
  a.k = (const _Float16*)k;
  a.vt = (const _Float16*)vt;
  a.o = (_Float16*)out;
  a.ldq = ldq;
  a.ldk = ldk;
  a.ldo = ldo;
  a.vt_ld = vt_ld;
  a.vt_row = vt_row;
  a.rows = rows;
  a.S = S;
  a.L = L;
  a.heads = heads;
  a.dh = dh;
  a.scale = scale;
  NV_HIP_TRY(attn_launch(a, (hipStream_t)stream));
  return NV_OK;
}
