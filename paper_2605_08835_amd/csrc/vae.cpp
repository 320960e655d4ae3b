// Host runtime of the VAE decoder: manifest, weight packing, the stage list
// VAE Chunking partitions, workspace planning and the launch sequence of a
// stage range.  The convolutions, GroupNorms and linears run on the UNet
// step's kernels (implicit-GEMM conv, GroupNorm statistics/apply); the
// decoder's own input, softmax and image write-out kernels are in vae_kernels.hip.
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <string>
#include <vector>

#include "kernels.h"
#include "manifest.h"
#include "synerdiff_vae.h"

namespace sd {
extern thread_local std::string g_err;

hipError_t launch_vae_input(DType dt, const float* lat, const float* w, const float* b, float inv_scale, void* y,
                            int n, int lc, int hw, int cpad, hipStream_t s);
hipError_t launch_softmax_rows(DType dt, const float* S, void* P, long rows, int cols, float scale, hipStream_t s);
hipError_t launch_image_out(const float* y, float* img, int n, int hw, int ld, int oc, hipStream_t s);

namespace {

sd_status vfail(sd_status s, const std::string& m) {
  g_err = m;
  return s;
}

inline size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

inline uint16_t to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

constexpr float VAE_GN_EPS = 1e-6f;
constexpr int CPAD = 8;  // input channels padded for 16-byte loads

std::string vae_check(const sd_vae_config& c) {
  if (c.dtype != SD_F32 && c.dtype != SD_BF16) return "dtype must be SD_F32 or SD_BF16";
  if (c.latent_c < 1 || c.latent_c > 8) return "latent_c must be 1..8";
  if (c.n_levels < 1 || c.n_levels > 4) return "n_levels must be 1..4";
  if (c.latent_h < 1 || c.latent_w < 1) return "bad latent size";
  if (c.n_res < 0 || c.n_res > 8) return "n_res must be 0..8";
  if (c.gn_groups < 1) return "gn_groups must be >= 1";
  if (c.out_c < 1 || c.out_c > 4) return "out_c must be 1..4";
  if (c.max_images < 1) return "max_images must be >= 1";
  if (!(c.scaling > 0.f) || !std::isfinite(c.scaling)) return "scaling must be positive";
  for (int l = 0; l < c.n_levels; ++l)
    if (c.ch[l] < 32 || c.ch[l] % 32 || c.ch[l] % c.gn_groups || c.ch[l] > 1024)
      return "ch[] must be multiples of 32 and of gn_groups, <= 1024";
  if ((long)c.latent_h * c.latent_w > 8192) return "latent_h * latent_w must be <= 8192 (mid attention)";
  const long Ho = (long)c.latent_h << (c.n_levels - 1), Wo = (long)c.latent_w << (c.n_levels - 1);
  if ((long)c.max_images * Ho * Wo * 1024 >= (1L << 31)) return "max_images x output pixels x width too large";
  return "";
}

struct VBuilder {
  std::vector<Param> P;
  size_t off = 0;
  void add(const std::string& n, std::vector<int64_t> s) {
    size_t k = 1;
    for (auto v : s) k *= (size_t)v;
    P.push_back(Param{n, std::move(s), off, k});
    off += k;
  }
  void res(const std::string& p, int ci, int co) {
    add(p + ".norm1.g", {ci});
    add(p + ".norm1.b", {ci});
    add(p + ".conv1.w", {co, ci, 3, 3});
    add(p + ".conv1.b", {co});
    add(p + ".norm2.g", {co});
    add(p + ".norm2.b", {co});
    add(p + ".conv2.w", {co, co, 3, 3});
    add(p + ".conv2.b", {co});
    if (ci != co) {
      add(p + ".skip.w", {co, ci});
      add(p + ".skip.b", {co});
    }
  }
};

// Parameters in load order: post_quant, conv_in, mid (res0, attn, res1),
// up levels from the widest, out.
std::vector<Param> vae_manifest(const sd_vae_config& c) {
  VBuilder b;
  const int lc = c.latent_c, nl = c.n_levels, top = c.ch[nl - 1];
  b.add("post_quant.w", {lc, lc});
  b.add("post_quant.b", {lc});
  b.add("conv_in.w", {top, lc, 3, 3});
  b.add("conv_in.b", {top});
  b.res("mid.res0", top, top);
  b.add("mid.attn.norm.g", {top});
  b.add("mid.attn.norm.b", {top});
  for (const char* p : {"q", "k", "v", "o"}) {
    b.add(std::string("mid.attn.") + p + ".w", {top, top});
    b.add(std::string("mid.attn.") + p + ".b", {top});
  }
  b.res("mid.res1", top, top);
  int cur = top;
  for (int i = 0; i < nl; ++i) {
    const int lvl = nl - 1 - i;
    for (int j = 0; j <= c.n_res; ++j) {
      b.res("up" + std::to_string(i) + ".res" + std::to_string(j), cur, c.ch[lvl]);
      cur = c.ch[lvl];
    }
    if (lvl != 0) {
      b.add("up" + std::to_string(i) + ".up.w", {cur, cur, 3, 3});
      b.add("up" + std::to_string(i) + ".up.b", {cur});
    }
  }
  b.add("out.norm.g", {c.ch[0]});
  b.add("out.norm.b", {c.ch[0]});
  b.add("out.conv.w", {c.out_c, c.ch[0], 3, 3});
  b.add("out.conv.b", {c.out_c});
  return b.P;
}

enum VKind { V_IN, V_RES, V_ATTN, V_UP, V_OUT };
enum VRole { VR_X0, VR_A, VR_B, VR_N, VR_U, VR_GNP, VR_GNS, VR_GNH, VR_Q, VR_K, VR_VT, VR_S, VR_P, VR_O, VR_Y, VR_SPLIT };

struct VConv {
  size_t w = 0, b = 0;
  int cin = 0, cout = 0, K = 0;
};

struct VStage {
  VKind kind;
  std::string name;
  int H, W, cin, cout;  // input size (upsampling doubles it) and widths
  int in_role, out_role;
  // parameters (packed offsets)
  size_t n1g = 0, n1b = 0, n2g = 0, n2b = 0;
  VConv c1, c2;  // RES: conv1, conv2 (+ 1x1 skip as extra K); UP / IN / OUT: c1
  bool skip = false;
  size_t pqw = 0, pqb = 0;                          // IN: post-quant (fp32)
  size_t ag = 0, ab = 0, aq = 0, aqb = 0, ak = 0, av = 0, ao = 0, aob = 0;  // ATTN
  double flop = 0;  // per image
};

enum PK { PK_ACT, PK_F32, PK_CONV3, PK_CONV3_SKIP, PK_F32_SUM, PK_VFOLD, PK_PAD_F32 };
struct VJob {
  PK kind;
  size_t dst;
  std::vector<std::string> names;
  int a = 0, b = 0;  // PK_CONV3*: cin_pad and (b > 0) the padded output rows; PK_PAD_F32: padded length
};

}  // namespace
}  // namespace sd

struct sd_vae {
  sd_vae_config cfg;
  sd::DType dt;
  int esz;
  uint8_t* wdev = nullptr;
  uint8_t* ws = nullptr;
  size_t wtotal = 0, wsbytes = 0;
  std::vector<sd::Param> manifest;
  std::vector<sd::VJob> jobs;
  std::vector<sd::VStage> stages;
  std::map<int, size_t> need, off;
  int next_stage = 0;  // chunked decode: the stage the next call must start at (0 = any)
  int run_n = 0;       // ... and its image count
};

namespace sd {
namespace {

size_t wal(sd_vae* h, size_t bytes) {
  const size_t o = al256(h->wtotal);
  h->wtotal = o + bytes;
  return o;
}
size_t jf32(sd_vae* h, std::vector<std::string> n, size_t numel, PK k = PK_F32) {
  const size_t d = wal(h, numel * 4);
  h->jobs.push_back(VJob{k, d, std::move(n)});
  return d;
}
size_t jact(sd_vae* h, std::vector<std::string> n, size_t numel) {
  const size_t d = wal(h, numel * h->esz);
  h->jobs.push_back(VJob{PK_ACT, d, std::move(n)});
  return d;
}
VConv conv3(sd_vae* h, const std::string& p, int cin, int cout, int cin_pad) {
  VConv c;
  c.cin = cin_pad;
  c.cout = cout;
  c.K = 9 * cin_pad;
  c.w = wal(h, (size_t)cout * c.K * h->esz);
  h->jobs.push_back(VJob{PK_CONV3, c.w, {p + ".w"}, cin_pad});
  c.b = jf32(h, {p + ".b"}, cout);
  return c;
}

double conv_flop(int H, int W, int cout, int K) { return 2.0 * H * W * cout * K; }

void build(sd_vae* h) {
  const sd_vae_config& c = h->cfg;
  const int nl = c.n_levels, top = c.ch[nl - 1];
  int H = c.latent_h, W = c.latent_w;
  int role = VR_A;
  auto flip = [&]() {
    const int o = role == VR_A ? VR_B : VR_A;
    return o;
  };
  {  // in
    VStage s{V_IN, "in", H, W, c.latent_c, top, VR_X0, VR_A};
    s.pqw = jf32(h, {"post_quant.w"}, (size_t)c.latent_c * c.latent_c);
    s.pqb = jf32(h, {"post_quant.b"}, c.latent_c);
    s.c1 = conv3(h, "conv_in", c.latent_c, top, CPAD);
    s.flop = 2.0 * H * W * c.latent_c * c.latent_c + conv_flop(H, W, top, 9 * c.latent_c);
    h->stages.push_back(s);
  }
  auto res = [&](const std::string& p, int ci, int co) {
    VStage s{V_RES, p, H, W, ci, co, role, flip()};
    s.n1g = jf32(h, {p + ".norm1.g"}, ci);
    s.n1b = jf32(h, {p + ".norm1.b"}, ci);
    s.c1 = conv3(h, p + ".conv1", ci, co, ci);
    s.n2g = jf32(h, {p + ".norm2.g"}, co);
    s.n2b = jf32(h, {p + ".norm2.b"}, co);
    s.skip = ci != co;
    s.c2.cin = co;
    s.c2.cout = co;
    s.c2.K = 9 * co + (s.skip ? ci : 0);
    s.c2.w = wal(h, (size_t)co * s.c2.K * h->esz);
    if (s.skip) {
      h->jobs.push_back(VJob{PK_CONV3_SKIP, s.c2.w, {p + ".conv2.w", p + ".skip.w"}, co});
      s.c2.b = jf32(h, {p + ".conv2.b", p + ".skip.b"}, co, PK_F32_SUM);
    } else {
      h->jobs.push_back(VJob{PK_CONV3, s.c2.w, {p + ".conv2.w"}, co});
      s.c2.b = jf32(h, {p + ".conv2.b"}, co);
    }
    s.flop = conv_flop(H, W, co, 9 * ci) + conv_flop(H, W, co, s.c2.K);
    h->stages.push_back(s);
    role = s.out_role;
  };
  res("mid.res0", top, top);
  {
    VStage s{V_ATTN, "mid.attn", H, W, top, top, role, flip()};
    const size_t CC = (size_t)top * top;
    s.ag = jf32(h, {"mid.attn.norm.g"}, top);
    s.ab = jf32(h, {"mid.attn.norm.b"}, top);
    s.aq = jact(h, {"mid.attn.q.w"}, CC);
    s.aqb = jf32(h, {"mid.attn.q.b"}, top);
    // keys need no bias: it shifts every score of a query by the same amount
    s.ak = jact(h, {"mid.attn.k.w"}, CC);
    // the value bias passes through the attention (rows of P sum to one)
    // and is folded into the output bias: b_o + W_o b_v
    s.av = jact(h, {"mid.attn.v.w"}, CC);
    s.ao = jact(h, {"mid.attn.o.w"}, CC);
    s.aob = wal(h, (size_t)top * 4);
    h->jobs.push_back(VJob{PK_VFOLD, s.aob, {"mid.attn.o.b", "mid.attn.o.w", "mid.attn.v.b"}});
    const double T = (double)H * W;
    s.flop = 4 * 2.0 * T * top * top + 2 * 2.0 * T * T * top;
    h->stages.push_back(s);
    role = s.out_role;
  }
  res("mid.res1", top, top);
  int cur = top;
  for (int i = 0; i < nl; ++i) {
    const int lvl = nl - 1 - i;
    for (int j = 0; j <= c.n_res; ++j) {
      res("up" + std::to_string(i) + ".res" + std::to_string(j), cur, c.ch[lvl]);
      cur = c.ch[lvl];
    }
    if (lvl != 0) {
      const std::string p = "up" + std::to_string(i) + ".up";
      VStage s{V_UP, p, H, W, cur, cur, role, flip()};
      s.c1 = conv3(h, p, cur, cur, cur);
      s.flop = conv_flop(2 * H, 2 * W, cur, 9 * cur);
      h->stages.push_back(s);
      role = s.out_role;
      H *= 2;
      W *= 2;
    }
  }
  {
    VStage s{V_OUT, "out", H, W, c.ch[0], c.out_c, role, VR_Y};
    s.n1g = jf32(h, {"out.norm.g"}, c.ch[0]);
    s.n1b = jf32(h, {"out.norm.b"}, c.ch[0]);
    // conv_out padded to 4 output channels (zero rows) for 8-byte stores
    s.c1.cin = c.ch[0];
    s.c1.cout = 4;
    s.c1.K = 9 * c.ch[0];
    s.c1.w = wal(h, (size_t)4 * s.c1.K * h->esz);
    h->jobs.push_back(VJob{PK_CONV3, s.c1.w, {"out.conv.w"}, c.ch[0], 4});
    s.c1.b = wal(h, 4 * 4);
    h->jobs.push_back(VJob{PK_PAD_F32, s.c1.b, {"out.conv.b"}, 0, 4});
    s.flop = conv_flop(H, W, c.out_c, 9 * c.ch[0]);
    h->stages.push_back(s);
  }
}

// ------------------------------------------------------------- execution
struct VRun {
  sd_vae* h;
  bool dry;
  hipStream_t s;
  int n;
  hipError_t err = hipSuccess;
  const char* where = "";

  void* buf(int role, size_t bytes) {
    if (dry) {
      size_t& v = h->need[role];
      v = std::max(v, bytes);
      return nullptr;
    }
    return h->ws + h->off.at(role);
  }
  const uint8_t* Wp(size_t o) const { return h->wdev + o; }
  const float* Wf(size_t o) const { return reinterpret_cast<const float*>(h->wdev + o); }
  bool ok(hipError_t e, const char* w) {
    if (e != hipSuccess && err == hipSuccess) {
      err = e;
      where = w;
    }
    return err == hipSuccess;
  }

  static ASeg seg(const void* x, int c, const void* x1, int c1, int ks, int up, int Hi, int Wi) {
    ASeg a;
    memset(&a, 0, sizeof(a));
    a.src0 = x;
    a.src1 = x1;
    a.c0 = c;
    a.c1 = c1;
    a.cin = c + c1;
    a.ks = ks;
    a.stride = 1;
    a.up = up;
    a.Hi = Hi;
    a.Wi = Wi;
    a.Ho = up ? 2 * Hi : Hi;
    a.Wo = up ? 2 * Wi : Wi;
    a.K = ks * ks * a.cin;
    return a;
  }
  static ASeg lin(const void* x, int K, long M) { return seg(x, K, nullptr, 0, 1, 0, 1, (int)M); }
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
  void gemm(const ASeg& s0, const ASeg* s1, const void* B, int ldb, int N, const Epi& e, long M, const char* w) {
    if (err) return;
    GemmArgs a;
    memset(&a, 0, sizeof(a));
    a.seg[0] = s0;
    if (s1) a.seg[1] = *s1;
    a.M = (int)M;
    a.N = N;
    a.K = s0.K + (s1 ? s1->K : 0);
    a.B = B;
    a.ldb = ldb;
    a.epi = e;
    a.ksplit = h->dt == BF16 ? gemm_ksplit(a) : 1;
    if (a.ksplit > 1) a.partial = (float*)buf(VR_SPLIT, (size_t)a.ksplit * a.M * N * 4);
    if (dry) return;
    ok(launch_gemm(h->dt, a, s), w);
  }
  // GroupNorm (+ SiLU) of x (n images, hw pixels, C channels) into VR_N.
  void* gn(const void* x, int C, int hw, size_t g, size_t b, int silu) {
    void* out = buf(VR_N, (size_t)n * hw * C * h->esz);
    if (groupnorm_fused_ok(h->dt, C, 0, hw, h->cfg.gn_groups)) {
      if (!dry && !err)
        ok(launch_groupnorm_fused(h->dt, x, C, nullptr, 0, n, hw, h->cfg.gn_groups, VAE_GN_EPS, Wf(g), Wf(b), silu,
                                  out, s),
           "vae groupnorm");
      return out;
    }
    float* part = (float*)buf(VR_GNP, groupnorm_partial_floats(n, hw, C) * 4);
    float* sc = (float*)buf(VR_GNS, (size_t)n * C * 4);
    float* sh = (float*)buf(VR_GNH, (size_t)n * C * 4);
    if (!dry && !err) {
      ok(launch_groupnorm_stats(h->dt, x, C, nullptr, 0, n, hw, h->cfg.gn_groups, VAE_GN_EPS, Wf(g), Wf(b), part, sc,
                                sh, s),
         "vae groupnorm");
      ok(launch_groupnorm_apply(h->dt, x, C, nullptr, 0, n, hw, sc, sh, silu, out, s), "vae groupnorm apply");
    }
    return out;
  }
  size_t act_bytes(int H, int W, int C) const { return (size_t)n * H * W * C * h->esz; }

  void stage(const VStage& st, const float* lat, float* img) {
    const int H = st.H, W = st.W, hw = H * W;
    switch (st.kind) {
      case V_IN: {
        void* x0 = buf(VR_X0, act_bytes(H, W, CPAD));
        void* out = buf(st.out_role, act_bytes(H, W, st.cout));
        if (!dry && !err)
          ok(launch_vae_input(h->dt, lat, Wf(st.pqw), Wf(st.pqb), 1.0f / h->cfg.scaling, x0, n, h->cfg.latent_c, hw,
                              CPAD, s),
             "vae input");
        gemm(seg(x0, CPAD, nullptr, 0, 3, 0, H, W), nullptr, Wp(st.c1.w), st.c1.K, st.cout,
             epi(out, st.cout, Wf(st.c1.b)), (long)n * hw, "vae conv_in");
        break;
      }
      case V_RES: {
        const void* x = buf(st.in_role, act_bytes(H, W, st.cin));
        void* out = buf(st.out_role, act_bytes(H, W, st.cout));
        void* u = buf(VR_U, act_bytes(H, W, st.cout));
        void* n1 = gn(x, st.cin, hw, st.n1g, st.n1b, 1);
        gemm(seg(n1, st.cin, nullptr, 0, 3, 0, H, W), nullptr, Wp(st.c1.w), st.c1.K, st.cout,
             epi(u, st.cout, Wf(st.c1.b)), (long)n * hw, "vae conv1");
        void* n2 = gn(u, st.cout, hw, st.n2g, st.n2b, 1);
        const ASeg a2 = seg(n2, st.cout, nullptr, 0, 3, 0, H, W);
        if (st.skip) {
          const ASeg sk = seg(x, st.cin, nullptr, 0, 1, 0, H, W);
          gemm(a2, &sk, Wp(st.c2.w), st.c2.K, st.cout, epi(out, st.cout, Wf(st.c2.b)), (long)n * hw, "vae conv2+skip");
        } else {
          gemm(a2, nullptr, Wp(st.c2.w), st.c2.K, st.cout, epi(out, st.cout, Wf(st.c2.b), x, st.cout), (long)n * hw,
               "vae conv2");
        }
        break;
      }
      case V_ATTN: {
        const int C = st.cin;
        const long T = hw;
        const void* x = buf(st.in_role, act_bytes(H, W, C));
        void* out = buf(st.out_role, act_bytes(H, W, C));
        void* xn = gn(x, C, hw, st.ag, st.ab, 0);
        void* q = buf(VR_Q, act_bytes(H, W, C));
        void* k = buf(VR_K, act_bytes(H, W, C));
        void* vt = buf(VR_VT, (size_t)C * T * h->esz);
        float* S = (float*)buf(VR_S, (size_t)T * T * 4);
        void* P = buf(VR_P, (size_t)T * T * h->esz);
        void* o = buf(VR_O, act_bytes(H, W, C));
        gemm(lin(xn, C, n * T), nullptr, Wp(st.aq), C, C, epi(q, C, Wf(st.aqb)), n * T, "vae attn q");
        gemm(lin(xn, C, n * T), nullptr, Wp(st.ak), C, C, epi(k, C, nullptr), n * T, "vae attn k");
        const auto at = [&](const void* p, long elems) -> const void* {
          return p ? (const uint8_t*)p + elems * h->esz : nullptr;
        };
        for (int i = 0; i < n && !err; ++i) {
          // V^T = W_v x^T (no bias): rows are channels, columns tokens
          gemm(lin(Wp(st.av), C, C), nullptr, at(xn, (long)i * T * C), C, (int)T, epi(vt, (int)T, nullptr), C,
               "vae attn v^T");
          Epi es = epi(S, (int)T, nullptr);
          es.out_f32 = 1;
          gemm(lin(at(q, (long)i * T * C), C, T), nullptr, at(k, (long)i * T * C), C, (int)T, es, T, "vae attn qk");
          if (!dry && !err) ok(launch_softmax_rows(h->dt, S, P, T, (int)T, 1.0f / sqrtf((float)C), s), "vae softmax");
          gemm(lin(P, (int)T, T), nullptr, vt, (int)T, C, epi((void*)at(o, (long)i * T * C), C, nullptr), T,
               "vae attn pv");
        }
        gemm(lin(o, C, n * T), nullptr, Wp(st.ao), C, C, epi(out, C, Wf(st.aob), x, C), n * T, "vae attn out");
        break;
      }
      case V_UP: {
        const void* x = buf(st.in_role, act_bytes(H, W, st.cin));
        void* out = buf(st.out_role, act_bytes(2 * H, 2 * W, st.cout));
        gemm(seg(x, st.cin, nullptr, 0, 3, 1, H, W), nullptr, Wp(st.c1.w), st.c1.K, st.cout,
             epi(out, st.cout, Wf(st.c1.b)), (long)n * 4 * hw, "vae upsample");
        break;
      }
      case V_OUT: {
        const void* x = buf(st.in_role, act_bytes(H, W, st.cin));
        void* xn = gn(x, st.cin, hw, st.n1g, st.n1b, 1);
        float* y = (float*)buf(VR_Y, (size_t)n * hw * 4 * 4);
        Epi e = epi(y, 4, Wf(st.c1.b));
        e.out_f32 = 1;
        gemm(seg(xn, st.cin, nullptr, 0, 3, 0, H, W), nullptr, Wp(st.c1.w), st.c1.K, 4, e, (long)n * hw,
             "vae conv_out");
        if (!dry && !err) ok(launch_image_out(y, img, n, hw, 4, st.cout, s), "vae image out");
        break;
      }
    }
  }
};

void plan(sd_vae* h) {
  VRun r{h, true, nullptr, h->cfg.max_images};
  for (const VStage& st : h->stages) r.stage(st, nullptr, nullptr);
  size_t o = 0;
  for (auto& kv : h->need) {
    h->off[kv.first] = o;
    o = al256(o + kv.second);
  }
  h->wsbytes = o;
}

sd_vae* skeleton(const sd_vae_config& c) {
  sd_vae* h = new sd_vae();
  h->cfg = c;
  h->dt = c.dtype == SD_BF16 ? BF16 : F32;
  h->esz = c.dtype == SD_BF16 ? 2 : 4;
  h->manifest = vae_manifest(c);
  build(h);
  plan(h);
  return h;
}

}  // namespace
}  // namespace sd

using namespace sd;

extern "C" {

sd_status synerdiff_vae_config_check(const sd_vae_config* cfg) {
  if (!cfg) return vfail(SD_ERR_INVALID_ARG, "cfg is NULL");
  const std::string why = vae_check(*cfg);
  return why.empty() ? SD_OK : vfail(SD_ERR_UNSUPPORTED, why);
}

int64_t synerdiff_vae_param_count(const sd_vae_config* cfg) {
  if (synerdiff_vae_config_check(cfg) != SD_OK) return -1;
  return (int64_t)vae_manifest(*cfg).size();
}

sd_status synerdiff_vae_param_info(const sd_vae_config* cfg, int64_t i, char* name, size_t cap, int64_t shape[4],
                                   int32_t* ndim) {
  const sd_status st = synerdiff_vae_config_check(cfg);
  if (st != SD_OK) return st;
  if (!name || !cap || !shape || !ndim) return vfail(SD_ERR_INVALID_ARG, "NULL output pointer");
  const auto m = vae_manifest(*cfg);
  if (i < 0 || i >= (int64_t)m.size()) return vfail(SD_ERR_INVALID_ARG, "parameter index out of range");
  const Param& p = m[(size_t)i];
  const size_t k = std::min(cap - 1, p.name.size());
  memcpy(name, p.name.data(), k);
  name[k] = 0;
  *ndim = (int32_t)p.shape.size();
  for (int d = 0; d < 4; ++d) shape[d] = d < (int)p.shape.size() ? p.shape[d] : 1;
  return SD_OK;
}

size_t synerdiff_vae_weights_bytes(const sd_vae_config* cfg) {
  if (synerdiff_vae_config_check(cfg) != SD_OK) return 0;
  sd_vae* h = skeleton(*cfg);
  const size_t n = al256(h->wtotal);
  delete h;
  return n;
}

size_t synerdiff_vae_workspace_bytes(const sd_vae_config* cfg) {
  if (synerdiff_vae_config_check(cfg) != SD_OK) return 0;
  sd_vae* h = skeleton(*cfg);
  const size_t n = h->wsbytes;
  delete h;
  return n;
}

sd_status synerdiff_vae_create(const sd_vae_config* cfg, void* dw, size_t wb, void* dws, size_t wsb, sd_vae** out) {
  if (!out) return vfail(SD_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  const sd_status st = synerdiff_vae_config_check(cfg);
  if (st != SD_OK) return st;
  if (!dw || !dws) return vfail(SD_ERR_INVALID_ARG, "NULL device buffer");
  if (((uintptr_t)dw & 255) || ((uintptr_t)dws & 255)) return vfail(SD_ERR_INVALID_ARG, "buffers must be 256-byte aligned");
  sd_vae* h = skeleton(*cfg);
  if (wb < al256(h->wtotal) || wsb < h->wsbytes) {
    delete h;
    return vfail(SD_ERR_WORKSPACE, "weight or workspace buffer too small");
  }
  h->wdev = (uint8_t*)dw;
  h->ws = (uint8_t*)dws;
  *out = h;
  return SD_OK;
}

sd_status synerdiff_vae_load_weights(sd_vae* h, const float* hp, size_t n_floats, void* stream) {
  if (!h || !hp) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  const Param& last = h->manifest.back();
  if (n_floats != last.offset + last.numel) return vfail(SD_ERR_INVALID_ARG, "n_floats does not match the manifest");
  std::map<std::string, const Param*> by;
  for (auto& p : h->manifest) by[p.name] = &p;
  std::vector<uint8_t> host(al256(h->wtotal), 0);
  const bool bf = h->dt == BF16;
  auto put = [&](size_t dst, size_t i, float v) {
    if (bf) {
      const uint16_t b = to_bf16(v);
      memcpy(&host[dst + i * 2], &b, 2);
    } else {
      memcpy(&host[dst + i * 4], &v, 4);
    }
  };
  auto putf = [&](size_t dst, size_t i, float v) { memcpy(&host[dst + i * 4], &v, 4); };
  for (const VJob& j : h->jobs) {
    std::vector<const Param*> src;
    for (auto& n : j.names) {
      auto it = by.find(n);
      if (it == by.end()) return vfail(SD_ERR_INVALID_ARG, "internal: missing parameter " + n);
      src.push_back(it->second);
    }
    const float* p0 = hp + src[0]->offset;
    switch (j.kind) {
      case PK_ACT:
        for (size_t i = 0; i < src[0]->numel; ++i) put(j.dst, i, p0[i]);
        break;
      case PK_F32:
        for (size_t i = 0; i < src[0]->numel; ++i) putf(j.dst, i, p0[i]);
        break;
      case PK_F32_SUM:
        for (size_t i = 0; i < src[0]->numel; ++i) putf(j.dst, i, p0[i] + hp[src[1]->offset + i]);
        break;
      case PK_PAD_F32:
        for (int i = 0; i < j.b; ++i) putf(j.dst, i, (size_t)i < src[0]->numel ? p0[i] : 0.f);
        break;
      case PK_VFOLD: {  // b_o + W_o b_v
        const size_t C = src[0]->numel;
        const float* wo = hp + src[1]->offset;
        const float* bv = hp + src[2]->offset;
        for (size_t o = 0; o < C; ++o) {
          double v = p0[o];
          for (size_t c = 0; c < C; ++c) v += (double)wo[o * C + c] * bv[c];
          putf(j.dst, o, (float)v);
        }
        break;
      }
      case PK_CONV3:
      case PK_CONV3_SKIP: {
        // [cout_pad][9 cin_pad (+ skip cin)]: tap-major, channel-minor
        const Param* w = src[0];
        const int cout = (int)w->shape[0], cin = (int)w->shape[1], cp = j.a;
        const int rows = j.b > 0 ? j.b : cout;
        const int ks = j.kind == PK_CONV3_SKIP ? (int)src[1]->shape[1] : 0;
        const int K = 9 * cp + ks;
        for (int o = 0; o < rows; ++o) {
          for (int t = 0; t < 9; ++t)
            for (int c = 0; c < cp; ++c) {
              const float v = (o < cout && c < cin) ? p0[((size_t)o * cin + c) * 9 + t] : 0.f;
              put(j.dst, (size_t)o * K + t * cp + c, v);
            }
          for (int c = 0; c < ks; ++c)
            put(j.dst, (size_t)o * K + 9 * cp + c, o < cout ? hp[src[1]->offset + (size_t)o * ks + c] : 0.f);
        }
        break;
      }
    }
  }
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(h->wdev, host.data(), host.size(), hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return vfail(SD_ERR_HIP, "weight upload failed");
  return SD_OK;
}

int32_t synerdiff_vae_stage_count(const sd_vae* h) { return h ? (int32_t)h->stages.size() : -1; }

sd_status synerdiff_vae_stage_name(const sd_vae* h, int32_t i, char* name, size_t cap) {
  if (!h || !name || !cap) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= (int32_t)h->stages.size()) return vfail(SD_ERR_INVALID_ARG, "stage index out of range");
  const std::string& n = h->stages[(size_t)i].name;
  const size_t k = std::min(cap - 1, n.size());
  memcpy(name, n.data(), k);
  name[k] = 0;
  return SD_OK;
}

sd_status synerdiff_vae_stage_flops(const sd_vae* h, int32_t i, double* flop) {
  if (!h || !flop) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i >= (int32_t)h->stages.size()) return vfail(SD_ERR_INVALID_ARG, "stage index out of range");
  *flop = h->stages[(size_t)i].flop;
  return SD_OK;
}

sd_status synerdiff_vae_run(sd_vae* h, int32_t n, const float* lat, int32_t begin, int32_t end, float* img,
                            void* stream) {
  if (!h) return vfail(SD_ERR_INVALID_ARG, "handle is NULL");
  const int ns = (int)h->stages.size();
  if (n < 1 || n > h->cfg.max_images) return vfail(SD_ERR_CAPACITY, "n must be 1..max_images");
  if (begin < 0 || end > ns || begin >= end) return vfail(SD_ERR_INVALID_ARG, "need 0 <= begin < end <= stage count");
  if (begin != 0 && (begin != h->next_stage || n != h->run_n))
    return vfail(SD_ERR_INVALID_ARG, "a chunk must start where the previous call ended, with the same n");
  if (begin == 0 && !lat) return vfail(SD_ERR_INVALID_ARG, "latents are NULL");
  if (end == ns && !img) return vfail(SD_ERR_INVALID_ARG, "image output is NULL");
  VRun r{h, false, (hipStream_t)stream, n};
  for (int i = begin; i < end && r.err == hipSuccess; ++i) r.stage(h->stages[(size_t)i], lat, img);
  if (r.err != hipSuccess) {
    h->next_stage = 0;
    return vfail(SD_ERR_HIP, std::string("HIP error in ") + r.where + ": " + hipGetErrorString(r.err));
  }
  h->next_stage = end == ns ? 0 : end;
  h->run_n = n;
  return SD_OK;
}

sd_status synerdiff_vae_activation(const sd_vae* h, int32_t i, int64_t* off, int32_t* H, int32_t* W, int32_t* C) {
  if (!h || !off || !H || !W || !C) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  if (i < 0 || i + 1 >= (int32_t)h->stages.size()) return vfail(SD_ERR_INVALID_ARG, "stage index out of range");
  const VStage& st = h->stages[(size_t)i];
  *off = (int64_t)h->off.at(st.out_role);
  *H = st.kind == V_UP ? 2 * st.H : st.H;
  *W = st.kind == V_UP ? 2 * st.W : st.W;
  *C = st.cout;
  return SD_OK;
}

void synerdiff_vae_destroy(sd_vae* h) { delete h; }

sd_status synerdiff_vae_chunk_plan(const double* cost, int32_t ns, int32_t c, int32_t* bounds) {
  if (!cost || !bounds) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  if (ns < 1 || c < 1 || c > ns) return vfail(SD_ERR_INVALID_ARG, "need 1 <= c <= n_stages");
  for (int i = 0; i < ns; ++i)
    if (!(cost[i] >= 0) || !std::isfinite(cost[i])) return vfail(SD_ERR_INVALID_ARG, "stage costs must be finite, >= 0");
  // best[k][i]: the smallest largest-chunk cost splitting stages [0, i) into k chunks
  std::vector<double> pre(ns + 1, 0.0);
  for (int i = 0; i < ns; ++i) pre[i + 1] = pre[i] + cost[i];
  const double INF = 1e300;
  std::vector<std::vector<double>> best(c + 1, std::vector<double>(ns + 1, INF));
  std::vector<std::vector<int>> arg(c + 1, std::vector<int>(ns + 1, -1));
  best[0][0] = 0.0;
  for (int k = 1; k <= c; ++k)
    for (int i = k; i <= ns; ++i)
      for (int j = k - 1; j < i; ++j) {  // last chunk [j, i)
        if (best[k - 1][j] >= INF) continue;
        const double v = std::max(best[k - 1][j], pre[i] - pre[j]);
        if (v < best[k][i]) {  // strict: ties keep the earliest boundary
          best[k][i] = v;
          arg[k][i] = j;
        }
      }
  bounds[c] = ns;
  for (int k = c, i = ns; k >= 1; --k) {
    i = arg[k][i];
    bounds[k - 1] = i;
  }
  return SD_OK;
}

sd_status synerdiff_chunk_cost(const double* t_u, const double* t_v, int32_t c, double T_u0, double T_v0,
                               double lambda, double* T_u, double* T_v, double* L) {
  if (!t_u || !t_v || !T_u || !T_v || !L) return vfail(SD_ERR_INVALID_ARG, "NULL argument");
  if (c < 1 || !(T_u0 > 0) || !(T_v0 > 0) || !(lambda >= 0 && lambda <= 1))
    return vfail(SD_ERR_INVALID_ARG, "need c >= 1, positive solo latencies, lambda in [0, 1]");
  double tu = 0.0, tv = 0.0;
  for (int i = 0; i < c; ++i) {
    const double m = std::max(t_u[i], t_v[i]);
    tu += m;
    tv += i + 1 < c ? m : t_v[i];
  }
  *T_u = tu;
  *T_v = tv;
  *L = lambda * (tu - T_u0) / T_u0 + (1.0 - lambda) * (tv - T_v0) / T_v0;
  return SD_OK;
}

}  // extern "C"
