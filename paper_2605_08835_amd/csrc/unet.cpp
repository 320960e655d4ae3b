// Host runtime of the UNet step: weight packing, workspace planning, the
// per-step row plan and the launch sequence.  All device work is enqueued on
// the caller's stream; the only host<->device traffic per step is one small
// H2D copy of the per-row scalars from a pinned staging ring.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <string.h>

#include <cmath>

#include <algorithm>
#include <functional>
#include <map>
#include <string>
#include <vector>

#include "kernels.h"
#include "manifest.h"
#include "synerdiff.h"

namespace sd {

thread_local std::string g_err;

static sd_status fail(sd_status s, const std::string& m) {
  g_err = m;
  return s;
}

static inline uint16_t f2bf(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFF) ? 0x40 : 0));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline float bf2f(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ------------------------------------------------------------------ layout
// P_*_GEGLU: rows of the GEGLU projection [a (4C) ; gate (4C)] reordered in
// blocks of 32 as [a 16t..16t+15 | gate 16t..16t+15] so that one 32-column
// MFMA tile holds matching value / gate columns.
// P_F32_VFOLD: self-attention output bias plus the output projection of the
// value bias that a folded LayerNorm's shift gives V (names: out bias, out
// weight, V weight, LN shift): b + W_o (W_v beta).  Attention rows of
// probabilities sum to one, so a bias on V passes through to the output.
// P_UPCONV (bf16): the 3x3 conv that follows a nearest-2x upsample, as four
// 2x2 convs on the small grid, one per output phase (py, px): tap (ty, tx)
// of phase (py, px) reads the input at (y + py - 1 + ty, x + px - 1 + tx)
// and its weight is the sum of the 3x3 taps (ky, kx) that land there,
// floor((py + ky - 1) / 2) = py - 1 + ty (likewise for x).  Layout
// [phase][cout][tap][cin].
enum PackKind { P_ACT, P_F32, P_F32_SUM, P_CONV3, P_CONV3_SKIP, P_ACT_GEGLU, P_F32_GEGLU, P_F32_VFOLD, P_UPCONV };
struct PackJob {
  PackKind kind;
  size_t dst;
  std::vector<std::string> names;
  int cin_pad;
  // P_ACT / P_ACT_GEGLU rows fed by a LayerNorm (bf16): each row becomes
  // w' = gamma w - mean_k(gamma w), so that x . w' = (x - mean(x)) . (gamma w)
  // for any input row x and the LN's mean subtraction happens inside the
  // product; the job also writes the bias with beta's product added
  // (fbias = bias + sum_k beta_k w_k; `bias` names the layer's bias, empty
  // for none).  The rounding to bf16 carries each element's error into the
  // next one, so a row's rounded elements still sum to ~0.
  std::string lng, lnb, bias;
  size_t fbias = 0;
  bool qk_only = false;  // [Q; K; V] rows: only the Q rows keep their folded bias
};

struct ConvW {
  size_t w = 0, b = 0;
  int cin = 0, cout = 0, K = 0;
  size_t wp = 0;  // upsampling convs: the four-phase weights (P_UPCONV), or 0
};
struct ResW {
  int cin = 0, cout = 0;
  size_t n1g = 0, n1b = 0, n2g = 0, n2b = 0;
  ConvW c1, c2;  // c2 holds [conv2 | skip] along K when the width changes
  bool skip = false;
  int tb_off = 0;
};
struct BlkW {
  size_t ln1g, ln1b, qkv, o1w, o1b, ln2g, ln2b, q2, kv2, o2w, o2b, ln3g, ln3b, f1w, f1b, f2w, f2b;
  // bf16: folded biases of the LN-fed projections
  size_t qkv_fb = 0, q2_fb = 0, f1_fb = 0;
};
struct TxW {
  int C = 0, heads = 0, d = 0;
  size_t ng = 0, nb = 0, piw = 0, pib = 0, pow = 0, pob = 0;
  std::vector<BlkW> blk;
};
struct LevelW {
  std::vector<ResW> res;
  std::vector<TxW> tx;  // empty when the level has no transformer
  bool has_conv = false;
  ConvW conv;  // downsample (down path) or upsample conv (up path)
};

// Workspace roles (buffers sized by a dry run at max capacity).
enum Role {
  R_X0, R_HA, R_HB, R_U, R_TZ, R_TX, R_TQ, R_TF, R_CTX, R_CKV, R_GNP, R_GNS, R_GNH,
  R_E, R_A, R_H1, R_TAU, R_T2, R_TB, R_EPS, R_SCAL, R_GNA, R_TV, R_CVT, R_SPLIT, R_LNS, R_SKIP0
};

}  // namespace sd

struct sd_unet {
  sd_unet_config cfg;
  sd::DType dt;
  int esz;  // activation element size
  uint8_t* wdev;
  size_t wbytes;
  uint8_t* ws;
  size_t wsbytes;
  std::vector<sd::Param> manifest;
  std::vector<sd::PackJob> jobs;
  size_t wtotal = 0;
  // network
  sd::ConvW conv_in;
  std::vector<sd::LevelW> down, up;
  sd::ResW mid0, mid1;
  std::vector<sd::TxW> midtx;
  size_t outg = 0, outb = 0;
  sd::ConvW conv_out;
  size_t t1w, t1b, t2w, t2b, a1w = 0, a1b = 0, a2w = 0, a2b = 0, tbw, tbb;
  int tb_total = 0;
  int cpad = 8;
  int n_skips = 0;
  // workspace
  std::map<int, size_t> need, off;
  size_t scal_bytes = 0;
  // profiling: one event after every launch; consecutive events bound it
  struct Rec {
    int kind;  // -1: start-of-step marker
    int layer;  // index into layer_names
    double flops, bytes;
    hipEvent_t ev;
  };
  bool prof = false;
  std::vector<hipEvent_t> pool;
  std::vector<Rec> recs;
  struct Tot {
    long launches = 0;
    double ms = 0, flops = 0, bytes = 0;
  } tot[16];
  std::map<std::string, int> layer_index;  // per-layer totals (name + shape)
  std::vector<std::string> layer_names;
  std::vector<Tot> ltot;
  // staging
  static constexpr int SLOTS = 8;
  uint8_t* pinned = nullptr;
  hipEvent_t ev[SLOTS] = {};
  int slot = 0;
};

namespace sd {

// ----------------------------------------------------------- weight arena
static size_t walloc(sd_unet* h, size_t bytes) {
  const size_t o = align256(h->wtotal);
  h->wtotal = o + bytes;
  return o;
}
static size_t job_act(sd_unet* h, std::vector<std::string> names, size_t numel) {
  const size_t d = walloc(h, numel * h->esz);
  h->jobs.push_back(PackJob{P_ACT, d, std::move(names), 0});
  return d;
}
// Marks the last pack job as fed by LayerNorm `ln` (bf16 weights only) and
// allocates its folded bias (rows fp32).
static void fold_ln(sd_unet* h, const std::string& ln, size_t rows, const std::string& bias, size_t& fb) {
  PackJob& j = h->jobs.back();
  j.lng = ln + ".g";
  j.lnb = ln + ".b";
  j.bias = bias;
  fb = j.fbias = walloc(h, rows * 4);
}

static size_t job_f32(sd_unet* h, std::vector<std::string> names, size_t numel, bool sum = false) {
  const size_t d = walloc(h, numel * 4);
  h->jobs.push_back(PackJob{sum ? P_F32_SUM : P_F32, d, std::move(names), 0});
  return d;
}

static ConvW conv3(sd_unet* h, const std::string& p, int cin, int cout, int cin_pad) {
  ConvW c;
  c.cin = cin_pad;
  c.cout = cout;
  c.K = 9 * cin_pad;
  c.w = walloc(h, (size_t)cout * c.K * h->esz);
  h->jobs.push_back(PackJob{P_CONV3, c.w, {p + ".w"}, cin_pad});
  c.b = job_f32(h, {p + ".b"}, cout);
  return c;
}

// Upsampling conv: the plain 3x3 weights, plus the four-phase form
// (P_UPCONV) where the GEMM takes it (bf16, width a multiple of 160).
static ConvW upconv(sd_unet* h, const std::string& p, int c) {
  ConvW w = conv3(h, p, c, c, c);
  if (h->dt == BF16 && c % 160 == 0) {
    w.wp = walloc(h, (size_t)16 * c * c * h->esz);
    h->jobs.push_back(PackJob{P_UPCONV, w.wp, {p + ".w"}, c});
  }
  return w;
}

static ResW resblock(sd_unet* h, const std::string& p, int cin, int cout, int& tb_off,
                     std::vector<std::string>& temb_names) {
  ResW r;
  r.cin = cin;
  r.cout = cout;
  r.skip = cin != cout;
  r.n1g = job_f32(h, {p + ".norm1.g"}, cin);
  r.n1b = job_f32(h, {p + ".norm1.b"}, cin);
  r.c1 = conv3(h, p + ".conv1", cin, cout, cin);
  r.n2g = job_f32(h, {p + ".norm2.g"}, cout);
  r.n2b = job_f32(h, {p + ".norm2.b"}, cout);
  r.c2.cin = cout;
  r.c2.cout = cout;
  r.c2.K = 9 * cout + (r.skip ? cin : 0);
  r.c2.w = walloc(h, (size_t)cout * r.c2.K * h->esz);
  if (r.skip) {
    h->jobs.push_back(PackJob{P_CONV3_SKIP, r.c2.w, {p + ".conv2.w", p + ".skip.w"}, cout});
    r.c2.b = job_f32(h, {p + ".conv2.b", p + ".skip.b"}, cout, true);
  } else {
    h->jobs.push_back(PackJob{P_CONV3, r.c2.w, {p + ".conv2.w"}, cout});
    r.c2.b = job_f32(h, {p + ".conv2.b"}, cout);
  }
  r.tb_off = tb_off;
  tb_off += cout;
  temb_names.push_back(p + ".temb");
  return r;
}

static TxW transformer(sd_unet* h, const std::string& p, int C, int depth) {
  const sd_unet_config& c = h->cfg;
  TxW t;
  t.C = C;
  t.heads = heads_at(c, C);
  t.d = C / t.heads;
  const size_t CC = (size_t)C * C;
  t.ng = job_f32(h, {p + ".norm.g"}, C);
  t.nb = job_f32(h, {p + ".norm.b"}, C);
  t.piw = job_act(h, {p + ".proj_in.w"}, CC);
  t.pib = job_f32(h, {p + ".proj_in.b"}, C);
  for (int j = 0; j < depth; ++j) {
    const std::string b = p + ".blk" + std::to_string(j);
    BlkW w;
    w.ln1g = job_f32(h, {b + ".ln1.g"}, C);
    w.ln1b = job_f32(h, {b + ".ln1.b"}, C);
    w.qkv = job_act(h, {b + ".attn1.q.w", b + ".attn1.k.w", b + ".attn1.v.w"}, 3 * CC);
    if (h->dt == BF16) {
      fold_ln(h, b + ".ln1", 3 * (size_t)C, "", w.qkv_fb);
      h->jobs.back().qk_only = true;
    }
    w.o1w = job_act(h, {b + ".attn1.o.w"}, CC);
    if (h->dt == BF16) {
      w.o1b = walloc(h, (size_t)C * 4);
      h->jobs.push_back(PackJob{P_F32_VFOLD, w.o1b, {b + ".attn1.o.b", b + ".attn1.o.w", b + ".attn1.v.w", b + ".ln1.b"}, 0});
    } else {
      w.o1b = job_f32(h, {b + ".attn1.o.b"}, C);
    }
    w.ln2g = job_f32(h, {b + ".ln2.g"}, C);
    w.ln2b = job_f32(h, {b + ".ln2.b"}, C);
    w.q2 = job_act(h, {b + ".attn2.q.w"}, CC);
    if (h->dt == BF16) fold_ln(h, b + ".ln2", C, "", w.q2_fb);
    w.kv2 = job_act(h, {b + ".attn2.k.w", b + ".attn2.v.w"}, (size_t)2 * C * c.ctx_dim);
    w.o2w = job_act(h, {b + ".attn2.o.w"}, CC);
    w.o2b = job_f32(h, {b + ".attn2.o.b"}, C);
    w.ln3g = job_f32(h, {b + ".ln3.g"}, C);
    w.ln3b = job_f32(h, {b + ".ln3.b"}, C);
    if (h->dt == BF16) {
      w.f1w = walloc(h, 8 * CC * h->esz);
      h->jobs.push_back(PackJob{P_ACT_GEGLU, w.f1w, {b + ".ff.w1"}, 0});
      fold_ln(h, b + ".ln3", 8 * (size_t)C, b + ".ff.b1", w.f1_fb);
      w.f1b = walloc(h, 8 * (size_t)C * 4);
      h->jobs.push_back(PackJob{P_F32_GEGLU, w.f1b, {b + ".ff.b1"}, 0});
    } else {
      w.f1w = job_act(h, {b + ".ff.w1"}, 8 * CC);
      w.f1b = job_f32(h, {b + ".ff.b1"}, 8 * C);
    }
    w.f2w = job_act(h, {b + ".ff.w2"}, 4 * CC);
    w.f2b = job_f32(h, {b + ".ff.b2"}, C);
    t.blk.push_back(w);
  }
  t.pow = job_act(h, {p + ".proj_out.w"}, CC);
  t.pob = job_f32(h, {p + ".proj_out.b"}, C);
  return t;
}

static void build_layout(sd_unet* h) {
  const sd_unet_config& c = h->cfg;
  const int td = c.temb_dim, nl = c.n_levels;
  h->t1w = job_act(h, {"time.lin1.w"}, (size_t)td * c.temb_in);
  h->t1b = job_f32(h, {"time.lin1.b"}, td);
  h->t2w = job_act(h, {"time.lin2.w"}, (size_t)td * td);
  h->t2b = job_f32(h, {"time.lin2.b"}, td);
  if (c.add_in) {
    h->a1w = job_act(h, {"add.lin1.w"}, (size_t)td * c.add_in);
    h->a1b = job_f32(h, {"add.lin1.b"}, td);
    h->a2w = job_act(h, {"add.lin2.w"}, (size_t)td * td);
    h->a2b = job_f32(h, {"add.lin2.b"}, td);
  }
  h->conv_in = conv3(h, "conv_in", c.latent_c, c.ch[0], h->cpad);
  int tb = 0;
  std::vector<std::string> temb;
  std::vector<int> skips{c.ch[0]};
  int cur = c.ch[0];
  h->down.resize(nl);
  for (int l = 0; l < nl; ++l) {
    const std::string p = "down" + std::to_string(l);
    for (int i = 0; i < c.n_res; ++i) {
      h->down[l].res.push_back(resblock(h, p + ".res" + std::to_string(i), cur, c.ch[l], tb, temb));
      cur = c.ch[l];
      if (c.tx_depth[l]) h->down[l].tx.push_back(transformer(h, p + ".tx" + std::to_string(i), cur, c.tx_depth[l]));
      skips.push_back(cur);
    }
    if (l != nl - 1) {
      h->down[l].has_conv = true;
      h->down[l].conv = conv3(h, p + ".down", cur, cur, cur);
      skips.push_back(cur);
    }
  }
  h->n_skips = (int)skips.size();
  h->mid0 = resblock(h, "mid.res0", cur, cur, tb, temb);
  if (c.mid_tx_depth) h->midtx.push_back(transformer(h, "mid.tx", cur, c.mid_tx_depth));
  h->mid1 = resblock(h, "mid.res1", cur, cur, tb, temb);
  h->up.resize(nl);
  for (int l = nl - 1; l >= 0; --l) {
    const std::string p = "up" + std::to_string(l);
    for (int i = 0; i <= c.n_res; ++i) {
      const int s = skips.back();
      skips.pop_back();
      h->up[l].res.push_back(resblock(h, p + ".res" + std::to_string(i), cur + s, c.ch[l], tb, temb));
      cur = c.ch[l];
      if (c.tx_depth[l]) h->up[l].tx.push_back(transformer(h, p + ".tx" + std::to_string(i), cur, c.tx_depth[l]));
    }
    if (l != 0) {
      h->up[l].has_conv = true;
      h->up[l].conv = upconv(h, p + ".up", cur);
    }
  }
  h->outg = job_f32(h, {"out.norm.g"}, c.ch[0]);
  h->outb = job_f32(h, {"out.norm.b"}, c.ch[0]);
  h->conv_out = conv3(h, "out.conv", c.ch[0], c.latent_c, c.ch[0]);
  h->tb_total = tb;
  std::vector<std::string> wn, bn;
  for (auto& n : temb) {
    wn.push_back(n + ".w");
    bn.push_back(n + ".b");
  }
  h->tbw = job_act(h, wn, (size_t)tb * td);
  h->tbb = job_f32(h, bn, tb);
}

// ------------------------------------------------------------- profiling
enum Kind { K_GEMM, K_ATTN, K_GN, K_LN, K_GEGLU, K_TIME, K_PACK, K_CFG, K_COPY, K_OUT, K_COUNT };
static const char* kKindName[K_COUNT] = {"gemm", "attention", "groupnorm", "layernorm", "geglu",
                                         "time_mlp", "pack", "cfg_ddim", "copy", "out_cfg_ddim"};

static hipEvent_t take_event(sd_unet* h) {
  if (!h->pool.empty()) {
    hipEvent_t e = h->pool.back();
    h->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
static void prof_mark(sd_unet* h, int kind, const char* name, double flops, double bytes, hipStream_t s) {
  hipEvent_t e = take_event(h);
  if (!e) return;
  if (hipEventRecord(e, s) != hipSuccess) {
    h->pool.push_back(e);
    return;
  }
  int layer = -1;
  if (kind >= 0 && name) {
    auto it = h->layer_index.find(name);
    if (it == h->layer_index.end()) {
      layer = (int)h->layer_names.size();
      h->layer_index.emplace(name, layer);
      h->layer_names.emplace_back(name);
      h->ltot.emplace_back();
    } else {
      layer = it->second;
    }
  }
  h->recs.push_back(sd_unet::Rec{kind, layer, flops, bytes, e});
}
static hipError_t prof_fold(sd_unet* h) {
  if (h->recs.empty()) return hipSuccess;
  hipError_t err = hipEventSynchronize(h->recs.back().ev);
  for (size_t i = 1; i < h->recs.size() && err == hipSuccess; ++i) {
    const auto& r = h->recs[i];
    if (r.kind < 0) continue;
    float ms = 0.f;
    err = hipEventElapsedTime(&ms, h->recs[i - 1].ev, r.ev);
    for (sd_unet::Tot* t : {&h->tot[r.kind], r.layer >= 0 ? &h->ltot[r.layer] : nullptr}) {
      if (!t) continue;
      t->launches++;
      t->ms += ms;
      t->flops += r.flops;
      t->bytes += r.bytes;
    }
  }
  for (auto& r : h->recs) h->pool.push_back(r.ev);
  h->recs.clear();
  return err;
}

// ------------------------------------------------------------- the step
struct Step {
  sd_unet* h;
  bool dry;
  hipStream_t s;
  int n_req, rows;
  // CFG pairs: until the first cross-attention a request's two rows see the
  // same latent, timestep and time embedding, so that prefix runs on the
  // conditional rows only (rows = n_req) and `expand` then copies them into
  // the unconditional rows (rows = full_rows).  Not with an added
  // embedding (SDXL's pooled text): there the two rows' time embeddings
  // differ from the start.  Buffers are sized for full_rows throughout.
  int full_rows = 0;
  std::function<void()> expand;
  const int* d_row_req = nullptr;  // device row plan: row_req[u] is the request of row u
  // Rows n_req .. full_rows - 1 of tensor t (row_bytes each) <- their requests' rows.
  void copy_rows(void* t, size_t row_bytes) {
    if (dry || err || rows >= full_rows) return;
    ok(launch_copy_rows(t, (long)row_bytes, n_req, full_rows - n_req, d_row_req + n_req, s), "cfg rows", K_COPY, 0,
       2.0 * (full_rows - n_req) * row_bytes);
  }
  hipError_t err = hipSuccess;
  const char* where = "";

  void* buf(int role, size_t bytes) {
    if (dry) {
      size_t& n = h->need[role];
      n = std::max(n, bytes);
      return nullptr;
    }
    return h->ws + h->off.at(role);
  }
  const uint8_t* W(size_t off) const { return h->wdev + off; }
  const float* Wf(size_t off) const { return reinterpret_cast<const float*>(h->wdev + off); }
  bool ok(hipError_t e, const char* w, int kind = K_COPY, double flops = 0, double bytes = 0) {
    if (e != hipSuccess && err == hipSuccess) {
      err = e;
      where = w;
    }
    if (err == hipSuccess && h->prof) prof_mark(h, kind, w, flops, bytes, s);
    return err == hipSuccess;
  }
  void* at(void* p, long elems) const { return p ? (uint8_t*)p + elems * h->esz : nullptr; }

  // GroupNorm statistics of [src0 | src1] -> (scale, shift) per (row, channel).
  void gn(const void* s0, int c0, const void* s1, int c1, int hw, float eps, size_t g, size_t b,
          float** sc, float** sh) {
    const int cin = c0 + c1;
    float* part = (float*)buf(R_GNP, groupnorm_partial_floats(rows, hw, cin) * 4);
    *sc = (float*)buf(R_GNS, (size_t)rows * cin * 4);
    *sh = (float*)buf(R_GNH, (size_t)rows * cin * 4);
    if (dry || err) return;
    ok(launch_groupnorm_stats(h->dt, s0, c0, s1, c1, rows, hw, h->cfg.gn_groups, eps, Wf(g), Wf(b), part,
                              *sc, *sh, s),
       "groupnorm", K_GN, 3.0 * rows * hw * cin, (double)rows * hw * cin * h->esz + 8.0 * rows * cin);
  }

  // GroupNorm (+ SiLU) of [src0 | src1] materialised as one [rows, hw, cin] tensor.
  void* gn_norm(const void* s0, int c0, const void* s1, int c1, int hw, float eps, size_t g, size_t b, int silu) {
    // images of 16x16 and smaller: one fused kernel (on the 640-channel
    // tensors at 32x32, which it would also take, the three passes are faster)
    if (hw <= 256 && groupnorm_fused_ok(h->dt, c0, c1, hw, h->cfg.gn_groups)) {
      const int cin = c0 + c1;
      void* out = buf(R_GNA, (size_t)rows * hw * cin * h->esz);
      if (dry || err) return out;
      ok(launch_groupnorm_fused(h->dt, s0, c0, s1, c1, rows, hw, h->cfg.gn_groups, eps, Wf(g), Wf(b), silu, out, s),
         "groupnorm fused", K_GN, (silu ? 9.0 : 5.0) * rows * hw * cin, 2.0 * rows * hw * cin * h->esz);
      return out;
    }
    float *sc, *sh;
    gn(s0, c0, s1, c1, hw, eps, g, b, &sc, &sh);
    const int cin = c0 + c1;
    void* out = buf(R_GNA, (size_t)rows * hw * cin * h->esz);
    if (dry || err) return out;
    ok(launch_groupnorm_apply(h->dt, s0, c0, s1, c1, rows, hw, sc, sh, silu, out, s), "groupnorm apply", K_GN,
       (silu ? 6.0 : 2.0) * rows * hw * cin, 2.0 * rows * hw * cin * h->esz);
    return out;
  }

  static ASeg seg(const void* s0, int c0, const void* s1, int c1, int ks, int stride, int up, int Hi,
                  int Wi, const float* sc, const float* sh, int silu) {
    ASeg a;
    a.src0 = s0;
    a.src1 = s1;
    a.scale = sc;
    a.shift = sh;
    a.c0 = c0;
    a.c1 = c1;
    a.cin = c0 + c1;
    a.ks = ks;
    a.stride = stride;
    a.up = up;
    a.Hi = Hi;
    a.Wi = Wi;
    a.Ho = up ? 2 * Hi : (stride == 2 ? (Hi - 1) / 2 + 1 : Hi);
    a.Wo = up ? 2 * Wi : (stride == 2 ? (Wi - 1) / 2 + 1 : Wi);
    a.K = ks * ks * a.cin;
    a.silu = silu;
    a.py = a.px = 0;
    return a;
  }
  static ASeg lin(const void* x, int K, long M) { return seg(x, K, nullptr, 0, 1, 1, 0, 1, (int)M, nullptr, nullptr, 0); }
  static Epi epi(void* out, int ldo, const float* bias, const void* resid = nullptr, int ldr = 0) {
    Epi e;
    memset(&e, 0, sizeof(e));
    e.out = out;
    e.ldo = ldo;
    e.bias = bias;
    e.resid = resid;
    e.ldr = ldr;
    e.hw = 1;
    return e;
  }
  // M defaults to rows * Ho * Wo (convolutions); linears pass it.  kalg
  // overrides the algorithmic K (conv_in's channel padding is not counted).
  void gemm(const ASeg& s0, const ASeg* s1, const void* B, int N, const Epi& e, const char* w, long M = -1,
            double kalg = -1) {
    if (err) return;
    GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.seg[0] = s0;
    if (s1) a.seg[1] = *s1;
    a.M = (int)(M >= 0 ? M : (long)rows * s0.Ho * s0.Wo);
    a.N = N;
    a.K = s0.K + (s1 ? s1->K : 0);
    a.B = B;
    a.ldb = a.K;
    a.epi = e;
    a.ksplit = h->dt == BF16 ? gemm_ksplit(a) : 1;
    if (a.ksplit > 1) a.partial = (float*)buf(R_SPLIT, (size_t)a.ksplit * a.M * N * 4);
    if (dry) return;
    const double K = kalg > 0 ? kalg : a.K;
    const double es = h->esz, outb = e.out_f32 ? 4 : es;
    auto seg_bytes = [&](const ASeg& g, long m) {
      return (g.Hi == 1 && g.Ho == 1) ? (double)m * g.cin * es : (double)rows * g.Hi * g.Wi * g.cin * es;
    };
    double bytes = seg_bytes(s0, a.M) + (s1 ? seg_bytes(*s1, a.M) : 0.0) + (double)N * a.K * es +
                   (double)a.M * N * outb + (e.resid ? (double)a.M * N * es : 0.0);
    char key[64];
    snprintf(key, sizeof(key), "%s %dx%dx%d", w, a.M, N, a.K);
    ok(launch_gemm(h->dt, a, s), h->prof ? key : w, K_GEMM, 2.0 * a.M * N * K, bytes);
  }
  // ResBlock on [src0 | src1] (H x W) -> out (cout channels).
  void resblock(const ResW& r, const void* s0, int c0, const void* s1, int c1, int H, int W_, void* out,
                const float* tb) {
    const int hw = H * W_, cin = c0 + c1;
    void* n1 = gn_norm(s0, c0, s1, c1, hw, 1e-5f, r.n1g, r.n1b, 1);
    void* u = buf(R_U, (size_t)rows * hw * r.cout * h->esz);
    Epi e1 = epi(u, r.cout, Wf(r.c1.b));
    e1.tbias = tb;
    e1.tb_ld = h->tb_total;
    e1.tb_off = r.tb_off;
    e1.hw = hw;
    gemm(seg(n1, cin, nullptr, 0, 3, 1, 0, H, W_, nullptr, nullptr, 0), nullptr, W(r.c1.w), r.cout, e1, "conv1");
    void* n2 = gn_norm(u, r.cout, nullptr, 0, hw, 1e-5f, r.n2g, r.n2b, 1);
    const ASeg a2 = seg(n2, r.cout, nullptr, 0, 3, 1, 0, H, W_, nullptr, nullptr, 0);
    if (r.skip) {
      const ASeg sk = seg(s0, c0, s1, c1, 1, 1, 0, H, W_, nullptr, nullptr, 0);
      gemm(a2, &sk, W(r.c2.w), r.cout, epi(out, r.cout, Wf(r.c2.b)), "conv2+skip");
    } else {
      gemm(a2, nullptr, W(r.c2.w), r.cout, epi(out, r.cout, Wf(r.c2.b), s0, r.cout), "conv2");
    }
  }

  // Transformer2D on h (H x W x C), in place.
  void transformer(const TxW& t, void* hbuf, int H, int W_, const void* ctx, const int* row_ctx) {
    const int hw = H * W_, C = t.C;
    long T = (long)rows * hw;
    const long Tmax = (long)std::max(rows, full_rows) * hw;  // buffer sizes
    const int L = h->cfg.ctx_len, D = h->cfg.ctx_dim;
    void* nh = gn_norm(hbuf, C, nullptr, 0, hw, 1e-6f, t.ng, t.nb, 0);
    void* z = buf(R_TZ, (size_t)Tmax * C * h->esz);
    void* x = buf(R_TX, (size_t)Tmax * C * h->esz);
    void* q = buf(R_TQ, (size_t)Tmax * 4 * C * h->esz);
    void* f = h->dt == BF16 ? nullptr : buf(R_TF, (size_t)Tmax * 8 * C * h->esz);
    void* ckv = buf(R_CKV, (size_t)(n_req + 1) * L * 2 * C * h->esz);
    const int Lp = (L + 7) / 8 * 8;
    void* vbuf = h->dt == BF16 ? buf(R_TV, (size_t)Tmax * C * h->esz) : nullptr;
    void* cvt = h->dt == BF16 ? buf(R_CVT, (size_t)(n_req + 1) * C * Lp * h->esz) : nullptr;
    gemm(lin(nh, C, T), nullptr, W(t.piw), C, epi(z, C, Wf(t.pib)), "proj_in", T);
    // bf16: the three LayerNorms are folded into the projections they feed
    // (mean subtraction and gain in the packed weights, shift in the bias,
    // the per-token 1/std applied in the epilogue), so only that scale is
    // computed here and the projections read z itself.  fp32: plain
    // LayerNorm into x.
    const bool fold = h->dt == BF16;
    float* lns = fold ? (float*)buf(R_LNS, (size_t)Tmax * 4) : nullptr;
    auto layernorm = [&](size_t g, size_t bb, const char* name) -> const void* {
      if (fold) {
        if (!dry && !err) ok(launch_layernorm_rstd(h->dt, z, lns, T, C, 1e-5f, s), name, K_LN, 4.0 * T * C, (double)T * C * h->esz + 4.0 * T);
        return z;
      }
      if (!dry && !err) ok(launch_layernorm(h->dt, z, x, T, C, Wf(g), Wf(bb), 1e-5f, s), name, K_LN, 8.0 * T * C, 2.0 * T * C * h->esz);
      return x;
    };
    auto lnepi = [&](Epi& e, size_t fb) {
      if (!fold) return;
      e.rowscale = lns;
      e.bias = Wf(fb);
    };
    for (const BlkW& b : t.blk) {
      const void* xin = layernorm(b.ln1g, b.ln1b, "ln1");
      // bf16: Q|K row-major [T, 2C], V transposed per image [rows][C][hw]
      // (the layout the attention kernel stages with 16-byte loads).
      const bool vt = h->dt == BF16;
      // bf16: queries leave the projection in base-2 logit units
      // (q * log2(e) / sqrt(d), one rounding), as the attention kernel takes them
      const float ql2 = 1.4426950408889634f / sqrtf((float)t.d);
      Epi eq = epi(q, vt ? 2 * C : 3 * C, nullptr);
      if (vt) {
        eq.qcols = C;
        eq.qscale = ql2;
        eq.vt_out = vbuf;
        eq.vt_col0 = 2 * C;
        eq.vt_hw = hw;
        eq.vt_ld = hw;
        eq.vt_img = (long)C * hw;
      }
      lnepi(eq, b.qkv_fb);
      gemm(lin(xin, C, T), nullptr, W(b.qkv), 3 * C, eq, "qkv", T);
      if (!dry && !err) {
        AttnArgs a;
        memset(&a, 0, sizeof(a));
        const long qld = vt ? 2 * C : 3 * C;
        a.q = q; a.q_ld = qld; a.q_img = (long)hw * qld;
        a.k = at(q, C); a.k_ld = qld; a.k_img = (long)hw * qld;
        if (vt) {
          a.v = vbuf; a.v_ld = hw; a.v_img = (long)C * hw; a.vt = 1;
        } else {
          a.v = at(q, 2 * C); a.v_ld = qld; a.v_img = (long)hw * qld;
        }
        a.kv_index = nullptr;
        a.o = x; a.o_ld = C; a.o_img = (long)hw * C;
        a.imgs = rows; a.heads = t.heads; a.d = t.d; a.Nq = hw; a.Nk = hw;
        a.scale = 1.0f / sqrtf((float)t.d);
        a.q_log2 = vt ? 1 : 0;
        char key[64];
        snprintf(key, sizeof(key), "self-attention %dx%d d%d", hw, hw, t.d);
        ok(launch_attention(h->dt, a, s), key, K_ATTN, 4.0 * rows * hw * (double)hw * C,
           4.0 * T * C * h->esz);
      }
      gemm(lin(x, C, T), nullptr, W(b.o1w), C, epi(z, C, Wf(b.o1b), z, C), "attn1.out", T);
      if (expand) {  // the rows diverge at the cross-attention: fill in the unconditional ones
        copy_rows(z, (size_t)hw * C * h->esz);
        expand();
        expand = nullptr;
        T = (long)rows * hw;
      }
      {
        const void* xin2 = layernorm(b.ln2g, b.ln2b, "ln2");
        Epi e2 = epi(q, C, nullptr);
        if (h->dt == BF16) {
          e2.qcols = C;
          e2.qscale = 1.4426950408889634f / sqrtf((float)t.d);
        }
        lnepi(e2, b.q2_fb);
        gemm(lin(xin2, C, T), nullptr, W(b.q2), C, e2, "attn2.q", T);
      }
      {
        const bool vt = h->dt == BF16;
        Epi ek = epi(ckv, vt ? C : 2 * C, nullptr);
        if (vt) {
          ek.vt_out = cvt;
          ek.vt_col0 = C;
          ek.vt_hw = L;
          ek.vt_ld = Lp;
          ek.vt_img = (long)C * Lp;
        }
        gemm(lin(ctx, D, (long)(n_req + 1) * L), nullptr, W(b.kv2), 2 * C, ek, "attn2.kv", (long)(n_req + 1) * L);
        if (!dry && !err) {
          AttnArgs a;
          memset(&a, 0, sizeof(a));
          const long kld = vt ? C : 2 * C;
          a.q = q; a.q_ld = C; a.q_img = (long)hw * C;
          a.k = ckv; a.k_ld = kld; a.k_img = (long)L * kld;
          if (vt) {
            a.v = cvt; a.v_ld = Lp; a.v_img = (long)C * Lp; a.vt = 1;
          } else {
            a.v = at(ckv, C); a.v_ld = kld; a.v_img = (long)L * kld;
          }
          a.kv_index = row_ctx;
          a.o = x; a.o_ld = C; a.o_img = (long)hw * C;
          a.imgs = rows; a.heads = t.heads; a.d = t.d; a.Nq = hw; a.Nk = L;
          a.scale = 1.0f / sqrtf((float)t.d);
          a.q_log2 = vt ? 1 : 0;
          char key[64];
          snprintf(key, sizeof(key), "cross-attention %dx%d d%d", hw, L, t.d);
          ok(launch_attention(h->dt, a, s), key, K_ATTN, 4.0 * rows * hw * (double)L * C,
             (2.0 * T * C + 2.0 * (n_req + 1) * L * C) * h->esz);
        }
      }
      gemm(lin(x, C, T), nullptr, W(b.o2w), C, epi(z, C, Wf(b.o2b), z, C), "attn2.out", T);
      const void* xin3 = layernorm(b.ln3g, b.ln3b, "ln3");
      if (h->dt == BF16) {  // GEGLU fused into the projection's epilogue
        Epi ef = epi(q, 4 * C, Wf(b.f1b));
        ef.geglu = 1;
        lnepi(ef, b.f1_fb);
        gemm(lin(xin3, C, T), nullptr, W(b.f1w), 8 * C, ef, "ff1+geglu", T);
      } else {
        gemm(lin(xin3, C, T), nullptr, W(b.f1w), 8 * C, epi(f, 8 * C, Wf(b.f1b)), "ff1", T);
        if (!dry && !err)
          ok(launch_geglu(h->dt, f, q, T, 4 * C, s), "geglu", K_GEGLU, 4.0 * T * 4 * C, 12.0 * T * C * h->esz);
      }
      gemm(lin(q, 4 * C, T), nullptr, W(b.f2w), C, epi(z, C, Wf(b.f2b), z, C), "ff2", T);
    }
    gemm(lin(z, C, T), nullptr, W(t.pow), C, epi(hbuf, C, Wf(t.pob), hbuf, C), "proj_out", T);
  }

  void run(const float* lat_in, const void* ctx_c, const void* ctx_u, const float* pool_c,
           const float* pool_u, float* lat_out, float* eps_out) {
    const sd_unet_config& c = h->cfg;
    const int nl = c.n_levels, td = c.temb_dim;
    int H = c.latent_h, Wd = c.latent_w;
    const int L = c.ctx_len, D = c.ctx_dim;
    // per-step scalars (uploaded by the caller of run)
    uint8_t* scal = (uint8_t*)buf(R_SCAL, h->scal_bytes);
    const int R = c.max_requests;
    const int* row_req = (const int*)(scal);
    const int* row_branch = (const int*)(scal + 4 * (2 * R));
    const int* row_ctx = (const int*)(scal + 4 * (4 * R));
    const float* row_t = (const float*)(scal + 4 * (6 * R));
    const int* req_row_u = (const int*)(scal + 4 * (8 * R));
    const float* req_coef = (const float*)(scal + 4 * (9 * R));
    const float* time_ids = (const float*)(scal + 4 * (12 * R));
    const int* req_order = (const int*)(scal + 4 * (12 * R + 64));

    if (!dry && h->prof) prof_mark(h, -1, nullptr, 0, 0, s);
    // contexts: [cond_0 .. cond_{n-1}, uncond]
    void* ctx = buf(R_CTX, (size_t)(n_req + 1) * L * D * h->esz);
    if (!dry && !err) {
      const size_t one = (size_t)L * D * h->esz;
      ok(hipMemcpyAsync(ctx, ctx_c, one * n_req, hipMemcpyDeviceToDevice, s), "ctx copy", K_COPY, 0, 2.0 * one * n_req);
      if (ctx_u) ok(hipMemcpyAsync((uint8_t*)ctx + one * n_req, ctx_u, one, hipMemcpyDeviceToDevice, s), "ctx copy", K_COPY, 0, 2.0 * one);
    }
    // time embedding -> per-row time bias of every ResBlock
    float* e = (float*)buf(R_E, (size_t)rows * c.temb_in * 4);
    float* a = c.add_in ? (float*)buf(R_A, (size_t)rows * c.add_in * 4) : nullptr;
    float* h1 = (float*)buf(R_H1, (size_t)rows * td * 4);
    float* tau = (float*)buf(R_TAU, (size_t)rows * td * 4);
    float* t2 = c.add_in ? (float*)buf(R_T2, (size_t)rows * td * 4) : nullptr;
    float* tb = (float*)buf(R_TB, (size_t)rows * h->tb_total * 4);
    if (!dry && !err) {
      ok(launch_time_inputs(row_t, rows, c.temb_in, e, pool_c, pool_u, row_req, row_branch, c.pooled_dim,
                            time_ids, c.n_time_ids, c.time_id_dim, a, s),
         "time inputs", K_TIME, 0, 4.0 * rows * (c.temb_in + c.add_in));
      ok(launch_linear_smallm(h->dt, e, rows, c.temb_in, W(h->t1w), Wf(h->t1b), nullptr, h1, td, 0, 1, s), "time.lin1", K_TIME,
         2.0 * rows * td * c.temb_in, (double)td * c.temb_in * h->esz);
      ok(launch_linear_smallm(h->dt, h1, rows, td, W(h->t2w), Wf(h->t2b), nullptr, tau, td, 0, 0, s), "time.lin2", K_TIME,
         2.0 * rows * td * td, (double)td * td * h->esz);
      if (c.add_in) {
        ok(launch_linear_smallm(h->dt, a, rows, c.add_in, W(h->a1w), Wf(h->a1b), nullptr, t2, td, 0, 1, s), "add.lin1", K_TIME,
           2.0 * rows * td * c.add_in, (double)td * c.add_in * h->esz);
        ok(launch_linear_smallm(h->dt, t2, rows, td, W(h->a2w), Wf(h->a2b), tau, tau, td, 0, 0, s), "add.lin2", K_TIME,
           2.0 * rows * td * td, (double)td * td * h->esz);
      }
      ok(launch_linear_smallm(h->dt, tau, rows, td, W(h->tbw), Wf(h->tbb), nullptr, tb, h->tb_total, 1, 0, s), "temb",
         K_TIME, 2.0 * rows * td * h->tb_total, (double)td * h->tb_total * h->esz + 4.0 * rows * h->tb_total);
    }
    // conditional rows only until the first cross-attention (see `expand`)
    full_rows = rows;
    d_row_req = row_req;
    if (rows > n_req && c.add_in == 0) rows = n_req;
    // pack + conv_in
    void* x0 = buf(R_X0, (size_t)full_rows * H * Wd * h->cpad * h->esz);
    if (!dry && !err)
      ok(launch_pack_latents(h->dt, lat_in, x0, rows, c.latent_c, H * Wd, h->cpad, row_req, s), "pack", K_PACK, 0,
         4.0 * n_req * c.latent_c * H * Wd + (double)rows * H * Wd * h->cpad * h->esz);
    std::vector<void*> skip(h->n_skips);
    std::vector<int> skipc(h->n_skips);
    std::vector<size_t> skiprow(h->n_skips);
    int k = 0;
    auto skipbuf = [&](int ch, int hh, int ww) {
      skipc[k] = ch;
      skiprow[k] = (size_t)hh * ww * ch * h->esz;
      skip[k] = buf(R_SKIP0 + k, (size_t)full_rows * skiprow[k]);
      return skip[k++];
    };
    // the live tensors at the first cross-attention are the skip stack so
    // far (the transformer's input is its last entry) and the transformer's z
    if (rows < full_rows) {
      expand = [&]() {
        for (int i = 0; i < k; ++i) copy_rows(skip[i], skiprow[i]);
        rows = full_rows;
      };
    }
    void* cur = skipbuf(c.ch[0], H, Wd);
    gemm(seg(x0, h->cpad, nullptr, 0, 3, 1, 0, H, Wd, nullptr, nullptr, 0), nullptr, W(h->conv_in.w), c.ch[0],
         epi(cur, c.ch[0], Wf(h->conv_in.b)), "conv_in", -1, 9.0 * c.latent_c);
    int curc = c.ch[0];
    for (int l = 0; l < nl; ++l) {
      const LevelW& lv = h->down[l];
      for (int i = 0; i < c.n_res; ++i) {
        const ResW& r = lv.res[i];
        void* o = skipbuf(r.cout, H, Wd);
        resblock(r, cur, curc, nullptr, 0, H, Wd, o, tb);
        if (!lv.tx.empty()) transformer(lv.tx[i], o, H, Wd, ctx, row_ctx);
        cur = o;
        curc = r.cout;
      }
      if (lv.has_conv) {
        const int Ho = H / 2, Wo = Wd / 2;
        void* o = skipbuf(curc, Ho, Wo);
        gemm(seg(cur, curc, nullptr, 0, 3, 2, 0, H, Wd, nullptr, nullptr, 0), nullptr, W(lv.conv.w), curc,
             epi(o, curc, Wf(lv.conv.b)), "downsample");
        cur = o;
        H = Ho;
        Wd = Wo;
      }
    }
    if (expand) {  // (no cross-attention on the down path)
      expand();
      expand = nullptr;
    }
    // hidden ping-pong buffers
    auto hbuf = [&](int role, int ch, int hh, int ww) { return buf(role, (size_t)rows * hh * ww * ch * h->esz); };
    void* ha = hbuf(R_HA, curc, H, Wd);
    resblock(h->mid0, cur, curc, nullptr, 0, H, Wd, ha, tb);
    if (!h->midtx.empty()) transformer(h->midtx[0], ha, H, Wd, ctx, row_ctx);
    void* hb = hbuf(R_HB, curc, H, Wd);
    resblock(h->mid1, ha, curc, nullptr, 0, H, Wd, hb, tb);
    cur = hb;
    int cur_role = R_HB;
    for (int l = nl - 1; l >= 0; --l) {
      const LevelW& lv = h->up[l];
      for (int i = 0; i <= c.n_res; ++i) {
        const ResW& r = lv.res[i];
        --k;
        const int nrole = cur_role == R_HA ? R_HB : R_HA;
        void* o = hbuf(nrole, r.cout, H, Wd);
        resblock(r, cur, curc, skip[k], skipc[k], H, Wd, o, tb);
        if (!lv.tx.empty()) transformer(lv.tx[i], o, H, Wd, ctx, row_ctx);
        cur = o;
        cur_role = nrole;
        curc = r.cout;
      }
      if (lv.has_conv) {
        const int nrole = cur_role == R_HA ? R_HB : R_HA;
        void* o = hbuf(nrole, curc, 2 * H, 2 * Wd);
        if (lv.conv.wp && H * Wd > 64) {
          // four 2x2 convs on the small grid, one per output phase (4/9 of
          // the 3x3's products; on 8x8 inputs the phases' grids are too
          // thin and the 3x3 form measured faster)
          for (int ph = 0; ph < 4; ++ph) {
            ASeg sg = seg(cur, curc, nullptr, 0, 2, 1, 0, H, Wd, nullptr, nullptr, 0);
            sg.py = ph >> 1;
            sg.px = ph & 1;
            Epi e = epi(o, curc, Wf(lv.conv.b));
            e.phase = 1 + ph;
            e.ph_h = H;
            e.ph_w = Wd;
            gemm(sg, nullptr, W(lv.conv.wp) + (size_t)ph * curc * 4 * curc * h->esz, curc, e, "upsample");
          }
        } else {
          gemm(seg(cur, curc, nullptr, 0, 3, 1, 1, H, Wd, nullptr, nullptr, 0), nullptr, W(lv.conv.w), curc,
               epi(o, curc, Wf(lv.conv.b)), "upsample");
        }
        cur = o;
        cur_role = nrole;
        H *= 2;
        Wd *= 2;
      }
    }
    // output: GN + SiLU, then the output conv, CFG combine and DDIM in one
    // kernel (bf16) or as conv (fp32 eps rows) + combine
    void* no = gn_norm(cur, curc, nullptr, 0, H * Wd, 1e-5f, h->outg, h->outb, 1);
    if (out_cfg_ddim_ok(h->dt, c.latent_c, H, Wd, curc)) {
      if (dry || err) return;
      OutArgs oa;
      memset(&oa, 0, sizeof(oa));
      oa.x = (const bf16_t*)no;
      oa.w = (const bf16_t*)W(h->conv_out.w);
      oa.bias = Wf(h->conv_out.b);
      oa.lat_in = lat_in;
      oa.lat_out = lat_out;
      oa.eps_out = eps_out;
      oa.req_row_u = req_row_u;
      oa.req_coef = req_coef;
      oa.order = req_order;
      oa.n_req = n_req;
      oa.H = H;
      oa.W = Wd;
      oa.C = curc;
      const double hw = (double)H * Wd;
      ok(launch_out_cfg_ddim(oa, s), "conv_out+cfg+ddim", K_OUT, 2.0 * rows * hw * 9.0 * curc * c.latent_c,
         (double)rows * hw * curc * h->esz + 4.0 * c.latent_c * hw * n_req * (2.0 + (eps_out ? 1.0 : 0.0)));
      return;
    }
    float* eps = (float*)buf(R_EPS, (size_t)rows * H * Wd * c.latent_c * 4);
    Epi eo = epi(eps, c.latent_c, Wf(h->conv_out.b));
    eo.out_f32 = 1;
    gemm(seg(no, curc, nullptr, 0, 3, 1, 0, H, Wd, nullptr, nullptr, 0), nullptr, W(h->conv_out.w), c.latent_c, eo,
         "conv_out");
    if (!dry && !err)
      ok(launch_cfg_ddim(eps, lat_in, lat_out, eps_out, n_req, c.latent_c, H * Wd, req_row_u, req_coef, s),
         "cfg+ddim", K_CFG, 4.0 * n_req * c.latent_c * H * Wd,
         4.0 * c.latent_c * H * Wd * (rows + 2.0 * n_req + (eps_out ? n_req : 0)));
  }
};

static void plan_workspace(sd_unet* h) {
  const int R = h->cfg.max_requests;
  h->scal_bytes = (size_t)4 * (13 * R + 64);
  Step st{h, true, nullptr, R, 2 * R};
  st.run(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
  size_t o = 0;
  for (auto& kv : h->need) {
    h->off[kv.first] = o;
    o = align256(o + kv.second);
  }
  h->wsbytes = o;
}

static bool get_config(const sd_unet_config* cfg, std::string& why) {
  if (!cfg) {
    why = "cfg is NULL";
    return false;
  }
  why = check_config(*cfg);
  return why.empty();
}

// Build a handle skeleton (layout + workspace plan) without device buffers.
static sd_unet* skeleton(const sd_unet_config* cfg) {
  sd_unet* h = new sd_unet();
  h->cfg = *cfg;
  h->dt = cfg->dtype == SD_BF16 ? BF16 : F32;
  h->esz = cfg->dtype == SD_BF16 ? 2 : 4;
  // conv_in's input channels padded to 32 in bf16 (a whole K stage per tap,
  // so it takes the direct-to-LDS GEMM; the padding adds only zero products),
  // to 8 in fp32
  h->cpad = h->dt == BF16 ? 32 : 8;
  h->manifest = build_manifest(*cfg);
  build_layout(h);
  plan_workspace(h);
  return h;
}

static bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uint8_t *pa = (const uint8_t*)a, *pb = (const uint8_t*)b;
  return pa < pb + nb && pb < pa + na;
}

}  // namespace sd

using namespace sd;

extern "C" {

int32_t synerdiff_abi_version(void) { return SYNERDIFF_ABI_VERSION; }

const char* synerdiff_last_error(void) { return g_err.c_str(); }

sd_status synerdiff_config_check(const sd_unet_config* cfg) {
  std::string why;
  if (!cfg) return fail(SD_ERR_INVALID_ARG, "cfg is NULL");
  if (!get_config(cfg, why)) return fail(SD_ERR_UNSUPPORTED, why);
  return SD_OK;
}

int64_t synerdiff_param_count(const sd_unet_config* cfg) {
  std::string why;
  if (!get_config(cfg, why)) {
    fail(SD_ERR_UNSUPPORTED, why);
    return -1;
  }
  return (int64_t)build_manifest(*cfg).size();
}

sd_status synerdiff_param_info(const sd_unet_config* cfg, int64_t i, char* name, size_t name_cap,
                               int64_t shape[4], int32_t* ndim) {
  std::string why;
  if (!get_config(cfg, why)) return fail(SD_ERR_UNSUPPORTED, why);
  if (!name || name_cap == 0 || !shape || !ndim) return fail(SD_ERR_INVALID_ARG, "NULL output pointer");
  const auto m = build_manifest(*cfg);
  if (i < 0 || i >= (int64_t)m.size()) return fail(SD_ERR_INVALID_ARG, "parameter index out of range");
  const Param& p = m[(size_t)i];
  const size_t n = std::min(name_cap - 1, p.name.size());
  memcpy(name, p.name.data(), n);
  name[n] = 0;
  *ndim = (int32_t)p.shape.size();
  for (int k = 0; k < 4; ++k) shape[k] = k < (int)p.shape.size() ? p.shape[k] : 1;
  return SD_OK;
}

size_t synerdiff_weights_bytes(const sd_unet_config* cfg) {
  std::string why;
  if (!get_config(cfg, why)) return 0;
  sd_unet* h = skeleton(cfg);
  const size_t n = align256(h->wtotal);
  delete h;
  return n;
}

size_t synerdiff_workspace_bytes(const sd_unet_config* cfg) {
  std::string why;
  if (!get_config(cfg, why)) return 0;
  sd_unet* h = skeleton(cfg);
  const size_t n = h->wsbytes;
  delete h;
  return n;
}

sd_status synerdiff_unet_create(const sd_unet_config* cfg, void* d_weights, size_t weights_bytes,
                                void* d_workspace, size_t workspace_bytes, sd_unet** out) {
  std::string why;
  if (!out) return fail(SD_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!cfg) return fail(SD_ERR_INVALID_ARG, "cfg is NULL");
  if (!get_config(cfg, why)) return fail(SD_ERR_UNSUPPORTED, why);
  if (!d_weights || !d_workspace) return fail(SD_ERR_INVALID_ARG, "NULL device buffer");
  if (((uintptr_t)d_weights & 255) || ((uintptr_t)d_workspace & 255))
    return fail(SD_ERR_INVALID_ARG, "device buffers must be 256-byte aligned");
  sd_unet* h = skeleton(cfg);
  if (weights_bytes < align256(h->wtotal) || workspace_bytes < h->wsbytes) {
    delete h;
    return fail(SD_ERR_WORKSPACE, "weight or workspace buffer too small");
  }
  h->wdev = (uint8_t*)d_weights;
  h->wbytes = weights_bytes;
  h->ws = (uint8_t*)d_workspace;
  *out = h;
  return SD_OK;
}

// The pinned staging ring and its events are created on the first step, so
// that creating a handle makes no HIP call.
static sd_status ensure_staging(sd_unet* h) {
  if (h->pinned) return SD_OK;
  if (hipHostMalloc((void**)&h->pinned, h->scal_bytes * sd_unet::SLOTS, hipHostMallocDefault) != hipSuccess) {
    h->pinned = nullptr;
    return fail(SD_ERR_HIP, "hipHostMalloc failed");
  }
  for (int i = 0; i < sd_unet::SLOTS; ++i)
    if (hipEventCreateWithFlags(&h->ev[i], hipEventDisableTiming) != hipSuccess)
      return fail(SD_ERR_HIP, "hipEventCreate failed");
  return SD_OK;
}

void synerdiff_unet_destroy(sd_unet* h) {
  if (!h) return;
  (void)prof_fold(h);
  for (hipEvent_t e : h->pool) (void)hipEventDestroy(e);
  for (int i = 0; i < sd_unet::SLOTS; ++i)
    if (h->ev[i]) {
      (void)hipEventSynchronize(h->ev[i]);
      (void)hipEventDestroy(h->ev[i]);
    }
  if (h->pinned) (void)hipHostFree(h->pinned);
  delete h;
}

sd_status synerdiff_load_weights(sd_unet* h, const float* hp, size_t n_floats, void* stream) {
  if (!h || !hp) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  const Param& last = h->manifest.back();
  if (n_floats != last.offset + last.numel) return fail(SD_ERR_INVALID_ARG, "n_floats does not match the manifest");
  std::map<std::string, const Param*> by;
  for (auto& p : h->manifest) by[p.name] = &p;
  std::vector<uint8_t> host(align256(h->wtotal), 0);
  const bool bf = h->dt == BF16;
  auto put_act = [&](size_t dst, size_t idx, float v) {
    if (bf) {
      const uint16_t b = f2bf(v);
      memcpy(&host[dst + idx * 2], &b, 2);
    } else {
      memcpy(&host[dst + idx * 4], &v, 4);
    }
  };
  for (const PackJob& j : h->jobs) {
    std::vector<const Param*> src;
    for (auto& n : j.names) {
      auto it = by.find(n);
      if (it == by.end()) return fail(SD_ERR_INVALID_ARG, "internal: missing parameter " + n);
      src.push_back(it->second);
    }
    if (!j.lng.empty()) {
      // LayerNorm-fed projection: source rows in packed order (GEGLU rows
      // reordered as below), each folded with the LN gain and shift.
      auto find = [&](const std::string& n) -> const Param* {
        auto it = by.find(n);
        return it == by.end() ? nullptr : it->second;
      };
      const Param* g = find(j.lng);
      const Param* be = find(j.lnb);
      const Param* bi = j.bias.empty() ? nullptr : find(j.bias);
      if (!g || !be || (!j.bias.empty() && !bi)) return fail(SD_ERR_INVALID_ARG, "internal: missing LN parameter");
      const size_t K = g->numel;
      std::vector<const float*> rowsrc;
      std::vector<float> rowbias;
      for (auto* p : src)
        for (size_t r = 0; r < p->numel / K; ++r) rowsrc.push_back(hp + p->offset + r * K);
      rowbias.assign(rowsrc.size(), 0.f);
      if (bi)
        for (size_t r = 0; r < rowsrc.size(); ++r) rowbias[r] = hp[bi->offset + r];
      if (j.kind == P_ACT_GEGLU) {
        const size_t rows8 = rowsrc.size(), half = rows8 / 2;
        std::vector<const float*> rs(rows8);
        std::vector<float> rb(rows8);
        for (size_t r = 0; r < rows8; ++r) {
          const size_t t = r / 32, u = r % 32;
          const size_t srow = u < 16 ? 16 * t + u : half + 16 * t + (u - 16);
          rs[r] = rowsrc[srow];
          rb[r] = rowbias[srow];
        }
        rowsrc.swap(rs);
        rowbias.swap(rb);
      }
      const float* gam = hp + g->offset;
      const float* bet = hp + be->offset;
      for (size_t r = 0; r < rowsrc.size(); ++r) {
        double mean = 0.0, fb = rowbias[r];
        for (size_t k = 0; k < K; ++k) {
          mean += (double)gam[k] * rowsrc[r][k];
          fb += (double)bet[k] * rowsrc[r][k];
        }
        mean /= (double)K;
        double carry = 0.0;  // rounding error carried to the next element
        for (size_t k = 0; k < K; ++k) {
          const double want = (double)gam[k] * rowsrc[r][k] - mean + carry;
          const float w = bf ? bf2f(f2bf((float)want)) : (float)want;
          put_act(j.dst, r * K + k, w);
          carry = want - (double)w;
        }
        // self-attention projections: keys need no bias (a shift of every
        // score of a query by the same q . b cancels in the softmax) and the
        // value bias moves to the output projection's bias (P_F32_VFOLD)
        const float fbf = (j.qk_only && r >= K) ? 0.f : (float)fb;
        memcpy(&host[j.fbias + r * 4], &fbf, 4);
      }
      continue;
    }
    switch (j.kind) {
      case P_ACT: {
        size_t o = 0;
        for (auto* p : src)
          for (size_t i = 0; i < p->numel; ++i) put_act(j.dst, o++, hp[p->offset + i]);
        break;
      }
      case P_F32: {
        size_t o = 0;
        for (auto* p : src) {
          memcpy(&host[j.dst + o * 4], hp + p->offset, p->numel * 4);
          o += p->numel;
        }
        break;
      }
      case P_ACT_GEGLU:
      case P_F32_GEGLU: {
        const Param* p = src[0];
        const size_t rows8 = (size_t)p->shape[0], half = rows8 / 2, cols = p->numel / rows8;
        for (size_t r = 0; r < rows8; ++r) {
          const size_t t = r / 32, u = r % 32;
          const size_t srow = u < 16 ? 16 * t + u : half + 16 * t + (u - 16);
          for (size_t k = 0; k < cols; ++k) {
            const float v = hp[p->offset + srow * cols + k];
            if (j.kind == P_ACT_GEGLU)
              put_act(j.dst, r * cols + k, v);
            else
              memcpy(&host[j.dst + (r * cols + k) * 4], &v, 4);
          }
        }
        break;
      }
      case P_F32_VFOLD: {
        const size_t C = src[0]->numel;
        std::vector<double> vb(C, 0.0);
        for (size_t c = 0; c < C; ++c)
          for (size_t k = 0; k < C; ++k) vb[c] += (double)hp[src[3]->offset + k] * hp[src[2]->offset + c * C + k];
        for (size_t n = 0; n < C; ++n) {
          double v = hp[src[0]->offset + n];
          for (size_t c = 0; c < C; ++c) v += (double)hp[src[1]->offset + n * C + c] * vb[c];
          const float f = (float)v;
          memcpy(&host[j.dst + n * 4], &f, 4);
        }
        break;
      }
      case P_F32_SUM: {
        for (size_t i = 0; i < src[0]->numel; ++i) {
          const float v = hp[src[0]->offset + i] + hp[src[1]->offset + i];
          memcpy(&host[j.dst + i * 4], &v, 4);
        }
        break;
      }
      case P_UPCONV: {
        const Param* w = src[0];
        const int cout = (int)w->shape[0], cin = (int)w->shape[1];
        const size_t K = 4 * (size_t)cin;
        auto src_off = [](int p, int k) { return (p + k + 1) / 2 - 1; };  // floor((p + k - 1) / 2)
        for (int ph = 0; ph < 4; ++ph) {
          const int py = ph >> 1, px = ph & 1;
          for (int o = 0; o < cout; ++o)
            for (int t = 0; t < 4; ++t) {
              const int dy = py - 1 + (t >> 1), dx = px - 1 + (t & 1);
              for (int c = 0; c < cin; ++c) {
                double v = 0.0;
                for (int ky = 0; ky < 3; ++ky)
                  for (int kx = 0; kx < 3; ++kx)
                    if (src_off(py, ky) == dy && src_off(px, kx) == dx)
                      v += hp[w->offset + ((size_t)o * cin + c) * 9 + ky * 3 + kx];
                put_act(j.dst, ((size_t)ph * cout + o) * K + (size_t)t * cin + c, (float)v);
              }
            }
        }
        break;
      }
      case P_CONV3:
      case P_CONV3_SKIP: {
        const Param* w = src[0];
        const int cout = (int)w->shape[0], cin = (int)w->shape[1];
        const int cp = j.cin_pad;
        const int K = 9 * cp + (j.kind == P_CONV3_SKIP ? (int)src[1]->shape[1] : 0);
        for (int o = 0; o < cout; ++o) {
          for (int tap = 0; tap < 9; ++tap)
            for (int c = 0; c < cp; ++c) {
              const float v = c < cin ? hp[w->offset + ((size_t)o * cin + c) * 9 + tap] : 0.f;
              put_act(j.dst, (size_t)o * K + tap * cp + c, v);
            }
          if (j.kind == P_CONV3_SKIP) {
            const Param* s = src[1];
            const int sc = (int)s->shape[1];
            for (int c = 0; c < sc; ++c) put_act(j.dst, (size_t)o * K + 9 * cp + c, hp[s->offset + (size_t)o * sc + c]);
          }
        }
        break;
      }
    }
  }
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(h->wdev, host.data(), host.size(), hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(SD_ERR_HIP, "weight upload failed");
  return SD_OK;
}

sd_status synerdiff_row_plan(int32_t n_req, const uint8_t* cfg_on, int32_t* row_req, int32_t* row_branch,
                             int32_t* req_row_u, int32_t* n_rows) {
  if (n_req < 0) return fail(SD_ERR_INVALID_ARG, "n_req < 0");
  if (n_req > 0 && (!cfg_on || !row_req || !row_branch || !req_row_u)) return fail(SD_ERR_INVALID_ARG, "NULL array");
  if (!n_rows) return fail(SD_ERR_INVALID_ARG, "n_rows is NULL");
  for (int r = 0; r < n_req; ++r)
    if (cfg_on[r] > 1) return fail(SD_ERR_INVALID_ARG, "cfg_on must be 0 or 1");
  int u = n_req;
  for (int r = 0; r < n_req; ++r) {
    row_req[r] = r;
    row_branch[r] = 0;
  }
  for (int r = 0; r < n_req; ++r) {
    if (cfg_on[r]) {
      row_req[u] = r;
      row_branch[u] = 1;
      req_row_u[r] = u++;
    } else {
      req_row_u[r] = -1;
    }
  }
  *n_rows = u;
  return SD_OK;
}

sd_status synerdiff_alphas_cumprod(int32_t schedule, double out[1000]) {
  if (!out) return fail(SD_ERR_INVALID_ARG, "out is NULL");
  double acc = 1.0;
  for (int t = 0; t < 1000; ++t) {
    const double s = t / 999.0;
    double beta;
    if (schedule == SD_SCHED_LINEAR) {
      beta = 1e-4 + (0.02 - 1e-4) * s;
    } else if (schedule == SD_SCHED_SCALED_LINEAR) {
      const double a = sqrt(0.00085), b = sqrt(0.012);
      beta = (a + (b - a) * s) * (a + (b - a) * s);
    } else {
      return fail(SD_ERR_INVALID_ARG, "unknown schedule");
    }
    acc *= 1.0 - beta;
    out[t] = acc;
  }
  return SD_OK;
}

sd_status synerdiff_ddim_coef(const double* ac, int32_t t, int32_t t_prev, float out_AB[2]) {
  if (!ac || !out_AB) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (t < 0 || t > 999 || t_prev > 999 || t_prev >= t) return fail(SD_ERR_INVALID_ARG, "need 0 <= t_prev < t <= 999 or t_prev < 0");
  const double at = ac[t], ap = t_prev < 0 ? 1.0 : ac[t_prev];
  out_AB[0] = (float)sqrt(ap / at);
  out_AB[1] = (float)(sqrt(1.0 - ap) - sqrt(ap * (1.0 - at) / at));
  return SD_OK;
}

sd_status synerdiff_ddim_coef_v(const double* ac, int32_t t, int32_t t_prev, float out_AB[2]) {
  if (!ac || !out_AB) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (t < 0 || t > 999 || t_prev > 999 || t_prev >= t) return fail(SD_ERR_INVALID_ARG, "need 0 <= t_prev < t <= 999 or t_prev < 0");
  // x0 = sqrt(a) x - sqrt(1 - a) v, eps = sqrt(1 - a) x + sqrt(a) v,
  // x' = sqrt(ap) x0 + sqrt(1 - ap) eps
  const double a = ac[t], ap = t_prev < 0 ? 1.0 : ac[t_prev];
  out_AB[0] = (float)(sqrt(ap * a) + sqrt((1.0 - ap) * (1.0 - a)));
  out_AB[1] = (float)(sqrt((1.0 - ap) * a) - sqrt(ap * (1.0 - a)));
  return SD_OK;
}

sd_status synerdiff_unet_create_shared(const sd_unet_config* cfg, const sd_unet* src, void* d_workspace,
                                       size_t workspace_bytes, sd_unet** out) {
  std::string why;
  if (!out) return fail(SD_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!cfg || !src) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (!get_config(cfg, why)) return fail(SD_ERR_UNSUPPORTED, why);
  sd_unet_config a = *cfg, b = src->cfg;
  a.latent_h = b.latent_h;
  a.latent_w = b.latent_w;
  a.max_requests = b.max_requests;
  if (memcmp(&a, &b, sizeof(a)) != 0)
    return fail(SD_ERR_INVALID_ARG, "configs may differ only in latent_h, latent_w and max_requests");
  if (!d_workspace || ((uintptr_t)d_workspace & 255))
    return fail(SD_ERR_INVALID_ARG, "workspace must be non-NULL and 256-byte aligned");
  sd_unet* h = skeleton(cfg);
  if (h->wtotal != src->wtotal) {
    delete h;
    return fail(SD_ERR_UNSUPPORTED, "internal: weight layouts differ");
  }
  if (workspace_bytes < h->wsbytes) {
    delete h;
    return fail(SD_ERR_WORKSPACE, "workspace buffer too small");
  }
  h->wdev = src->wdev;
  h->wbytes = src->wbytes;
  h->ws = (uint8_t*)d_workspace;
  *out = h;
  return SD_OK;
}

sd_status synerdiff_unet_step(sd_unet* h, int32_t n_req, const float* lat_in, const int32_t* ts,
                              const uint8_t* cfg_on, const float* guidance, const void* ctx_c,
                              const void* ctx_u, const float* pool_c, const float* pool_u,
                              const float* time_ids, const float* coef, float* lat_out, float* eps_out,
                              void* stream) {
  if (!h) return fail(SD_ERR_INVALID_ARG, "handle is NULL");
  if (n_req < 0) return fail(SD_ERR_INVALID_ARG, "n_req < 0");
  if (n_req == 0) return SD_OK;
  const sd_unet_config& c = h->cfg;
  if (n_req > c.max_requests) return fail(SD_ERR_CAPACITY, "n_req exceeds max_requests");
  if (!lat_in || !ts || !cfg_on || !ctx_c || !coef || !lat_out) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  int ncfg = 0;
  for (int r = 0; r < n_req; ++r) {
    if (ts[r] < 0 || ts[r] > 999) return fail(SD_ERR_INVALID_ARG, "timestep out of [0, 999]");
    if (cfg_on[r] > 1) return fail(SD_ERR_INVALID_ARG, "cfg_on must be 0 or 1");
    if (!std::isfinite(coef[2 * r]) || !std::isfinite(coef[2 * r + 1]))
      return fail(SD_ERR_INVALID_ARG, "non-finite sampler coefficient");
    if (cfg_on[r]) {
      ++ncfg;
      if (!guidance) return fail(SD_ERR_INVALID_ARG, "guidance is NULL");
      if (!std::isfinite(guidance[r])) return fail(SD_ERR_INVALID_ARG, "non-finite guidance");
    }
  }
  if (ncfg && !ctx_u) return fail(SD_ERR_INVALID_ARG, "ctx_uncond is NULL");
  if (c.add_in) {
    if (!pool_c || (ncfg && !pool_u) || (c.n_time_ids && !time_ids))
      return fail(SD_ERR_INVALID_ARG, "pooled / time_ids required for the added embedding");
  } else if (pool_c || pool_u) {
    return fail(SD_ERR_INVALID_ARG, "pooled inputs given but the config has no added embedding");
  }
  const size_t lat_bytes = (size_t)n_req * c.latent_c * c.latent_h * c.latent_w * 4;
  if (lat_out != lat_in && ranges_overlap(lat_out, lat_bytes, lat_in, lat_bytes))
    return fail(SD_ERR_INVALID_ARG, "latents_out partially overlaps latents_in");
  if (eps_out && (ranges_overlap(eps_out, lat_bytes, lat_in, lat_bytes) || ranges_overlap(eps_out, lat_bytes, lat_out, lat_bytes)))
    return fail(SD_ERR_INVALID_ARG, "eps_out overlaps the latents");

  // row plan + scalars into a pinned slot, one H2D copy
  if (ensure_staging(h) != SD_OK) return SD_ERR_HIP;
  const int R = c.max_requests;
  hipStream_t s = (hipStream_t)stream;
  const int slot = h->slot;
  h->slot = (h->slot + 1) % sd_unet::SLOTS;
  if (hipEventSynchronize(h->ev[slot]) != hipSuccess) return fail(SD_ERR_HIP, "staging event wait failed");
  uint8_t* p = h->pinned + h->scal_bytes * slot;
  memset(p, 0, h->scal_bytes);
  int32_t* row_req = (int32_t*)p;
  int32_t* row_branch = (int32_t*)(p + 4 * (2 * R));
  int32_t* row_ctx = (int32_t*)(p + 4 * (4 * R));
  float* row_t = (float*)(p + 4 * (6 * R));
  int32_t* req_row_u = (int32_t*)(p + 4 * (8 * R));
  float* req_coef = (float*)(p + 4 * (9 * R));
  float* tid = (float*)(p + 4 * (12 * R));
  int32_t* req_order = (int32_t*)(p + 4 * (12 * R + 64));
  int rows = 0;
  synerdiff_row_plan(n_req, cfg_on, row_req, row_branch, req_row_u, &rows);
  for (int i = 0; i < rows; ++i) {
    row_ctx[i] = row_branch[i] ? n_req : row_req[i];
    row_t[i] = (float)ts[row_req[i]];
  }
  for (int r = 0; r < n_req; ++r) {
    req_coef[3 * r] = coef[2 * r];
    req_coef[3 * r + 1] = coef[2 * r + 1];
    req_coef[3 * r + 2] = cfg_on[r] ? guidance[r] : 1.0f;
  }
  for (int i = 0; i < c.n_time_ids && time_ids; ++i) tid[i] = time_ids[i];
  {  // requests with two rows (the longer output blocks) are launched first
    int k = 0;
    for (int r = 0; r < n_req; ++r)
      if (cfg_on[r]) req_order[k++] = r;
    for (int r = 0; r < n_req; ++r)
      if (!cfg_on[r]) req_order[k++] = r;
  }
  if (hipMemcpyAsync(h->ws + h->off.at(R_SCAL), p, h->scal_bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipEventRecord(h->ev[slot], s) != hipSuccess)
    return fail(SD_ERR_HIP, "scalar upload failed");

  Step st{h, false, s, n_req, rows};
  st.run(lat_in, ctx_c, ctx_u, pool_c, pool_u, lat_out, eps_out);
  if (st.err != hipSuccess)
    return fail(SD_ERR_HIP, std::string("HIP error in ") + st.where + ": " + hipGetErrorString(st.err));
  return SD_OK;
}

sd_status synerdiff_profile(sd_unet* h, int32_t enable) {
  if (!h) return fail(SD_ERR_INVALID_ARG, "handle is NULL");
  h->prof = enable != 0;
  return SD_OK;
}

sd_status synerdiff_profile_read(sd_unet* h, sd_kernel_stat* out, int32_t cap, int32_t* n_out, int32_t reset) {
  if (!h || !n_out || (cap > 0 && !out)) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (prof_fold(h) != hipSuccess) return fail(SD_ERR_HIP, "profiling event query failed");
  int n = 0;
  for (int k = 0; k < K_COUNT; ++k) {
    if (!h->tot[k].launches) continue;
    if (n < cap) {
      sd_kernel_stat& o = out[n];
      memset(&o, 0, sizeof(o));
      strncpy(o.name, kKindName[k], sizeof(o.name) - 1);
      o.launches = h->tot[k].launches;
      o.ms = h->tot[k].ms;
      o.flop = h->tot[k].flops;
      o.bytes = h->tot[k].bytes;
    }
    ++n;
  }
  *n_out = n;
  if (reset)
    for (auto& t : h->tot) t = sd_unet::Tot();
  return SD_OK;
}

sd_status synerdiff_profile_read_layers(sd_unet* h, sd_layer_stat* out, int32_t cap, int32_t* n_out,
                                        int32_t reset) {
  if (!h || !n_out || (cap > 0 && !out)) return fail(SD_ERR_INVALID_ARG, "NULL argument");
  if (prof_fold(h) != hipSuccess) return fail(SD_ERR_HIP, "profiling event query failed");
  int n = 0;
  for (size_t i = 0; i < h->ltot.size(); ++i) {
    if (!h->ltot[i].launches) continue;
    if (n < cap) {
      sd_layer_stat& o = out[n];
      memset(&o, 0, sizeof(o));
      strncpy(o.name, h->layer_names[i].c_str(), sizeof(o.name) - 1);
      o.launches = h->ltot[i].launches;
      o.ms = h->ltot[i].ms;
      o.flop = h->ltot[i].flops;
      o.bytes = h->ltot[i].bytes;
    }
    ++n;
  }
  *n_out = n;
  if (reset)
    for (auto& t : h->ltot) t = sd_unet::Tot();
  return SD_OK;
}

}  // extern "C"
