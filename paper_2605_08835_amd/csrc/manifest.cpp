#include "manifest.h"

#include "kernels.h"

namespace sd {

namespace {

struct Builder {
  std::vector<Param> P;
  size_t off = 0;
  void add(const std::string& n, std::vector<int64_t> s) {
    size_t k = 1;
    for (auto v : s) k *= (size_t)v;
    P.push_back(Param{n, std::move(s), off, k});
    off += k;
  }
  void resblock(const std::string& p, int cin, int cout, int td) {
    add(p + ".norm1.g", {cin});
    add(p + ".norm1.b", {cin});
    add(p + ".conv1.w", {cout, cin, 3, 3});
    add(p + ".conv1.b", {cout});
    add(p + ".temb.w", {cout, td});
    add(p + ".temb.b", {cout});
    add(p + ".norm2.g", {cout});
    add(p + ".norm2.b", {cout});
    add(p + ".conv2.w", {cout, cout, 3, 3});
    add(p + ".conv2.b", {cout});
    if (cin != cout) {
      add(p + ".skip.w", {cout, cin});
      add(p + ".skip.b", {cout});
    }
  }
  void transformer(const std::string& p, int c, int depth, int ctx_dim) {
    add(p + ".norm.g", {c});
    add(p + ".norm.b", {c});
    add(p + ".proj_in.w", {c, c});
    add(p + ".proj_in.b", {c});
    for (int j = 0; j < depth; ++j) {
      const std::string b = p + ".blk" + std::to_string(j);
      add(b + ".ln1.g", {c});
      add(b + ".ln1.b", {c});
      add(b + ".attn1.q.w", {c, c});
      add(b + ".attn1.k.w", {c, c});
      add(b + ".attn1.v.w", {c, c});
      add(b + ".attn1.o.w", {c, c});
      add(b + ".attn1.o.b", {c});
      add(b + ".ln2.g", {c});
      add(b + ".ln2.b", {c});
      add(b + ".attn2.q.w", {c, c});
      add(b + ".attn2.k.w", {c, ctx_dim});
      add(b + ".attn2.v.w", {c, ctx_dim});
      add(b + ".attn2.o.w", {c, c});
      add(b + ".attn2.o.b", {c});
      add(b + ".ln3.g", {c});
      add(b + ".ln3.b", {c});
      add(b + ".ff.w1", {8 * c, c});
      add(b + ".ff.b1", {8 * c});
      add(b + ".ff.w2", {c, 4 * c});
      add(b + ".ff.b2", {c});
    }
    add(p + ".proj_out.w", {c, c});
    add(p + ".proj_out.b", {c});
  }
};

}  // namespace

std::vector<Param> build_manifest(const sd_unet_config& c) {
  Builder B;
  const int td = c.temb_dim, nl = c.n_levels;
  B.add("time.lin1.w", {td, c.temb_in});
  B.add("time.lin1.b", {td});
  B.add("time.lin2.w", {td, td});
  B.add("time.lin2.b", {td});
  if (c.add_in) {
    B.add("add.lin1.w", {td, c.add_in});
    B.add("add.lin1.b", {td});
    B.add("add.lin2.w", {td, td});
    B.add("add.lin2.b", {td});
  }
  B.add("conv_in.w", {c.ch[0], c.latent_c, 3, 3});
  B.add("conv_in.b", {c.ch[0]});
  std::vector<int> skips{c.ch[0]};
  int cur = c.ch[0];
  for (int l = 0; l < nl; ++l) {
    for (int i = 0; i < c.n_res; ++i) {
      const std::string p = "down" + std::to_string(l);
      B.resblock(p + ".res" + std::to_string(i), cur, c.ch[l], td);
      cur = c.ch[l];
      if (c.tx_depth[l]) B.transformer(p + ".tx" + std::to_string(i), cur, c.tx_depth[l], c.ctx_dim);
      skips.push_back(cur);
    }
    if (l != nl - 1) {
      B.add("down" + std::to_string(l) + ".down.w", {cur, cur, 3, 3});
      B.add("down" + std::to_string(l) + ".down.b", {cur});
      skips.push_back(cur);
    }
  }
  B.resblock("mid.res0", cur, cur, td);
  if (c.mid_tx_depth) B.transformer("mid.tx", cur, c.mid_tx_depth, c.ctx_dim);
  B.resblock("mid.res1", cur, cur, td);
  for (int l = nl - 1; l >= 0; --l) {
    const std::string p = "up" + std::to_string(l);
    for (int i = 0; i <= c.n_res; ++i) {
      const int s = skips.back();
      skips.pop_back();
      B.resblock(p + ".res" + std::to_string(i), cur + s, c.ch[l], td);
      cur = c.ch[l];
      if (c.tx_depth[l]) B.transformer(p + ".tx" + std::to_string(i), cur, c.tx_depth[l], c.ctx_dim);
    }
    if (l != 0) {
      B.add(p + ".up.w", {cur, cur, 3, 3});
      B.add(p + ".up.b", {cur});
    }
  }
  B.add("out.norm.g", {c.ch[0]});
  B.add("out.norm.b", {c.ch[0]});
  B.add("out.conv.w", {c.latent_c, c.ch[0], 3, 3});
  B.add("out.conv.b", {c.latent_c});
  return B.P;
}

std::string check_config(const sd_unet_config& c) {
  if (c.dtype != SD_F32 && c.dtype != SD_BF16) return "dtype must be SD_F32 or SD_BF16";
  if (c.latent_c < 1 || c.latent_c > 8) return "latent_c must be in [1, 8]";
  if (c.n_levels < 1 || c.n_levels > 4) return "n_levels must be in [1, 4]";
  if (c.latent_h < 1 || c.latent_w < 1) return "latent size must be positive";
  const int f = 1 << (c.n_levels - 1);
  if (c.latent_h % f || c.latent_w % f) return "latent size must be divisible by 2^(n_levels-1)";
  if (c.n_res < 1) return "n_res must be >= 1";
  if ((c.heads == 0) == (c.head_dim == 0)) return "exactly one of heads, head_dim must be non-zero";
  if (c.heads < 0 || c.head_dim < 0) return "heads / head_dim must be non-negative";
  if (c.gn_groups < 1) return "gn_groups must be >= 1";
  if (c.ctx_len < 1 || c.ctx_dim < 8 || c.ctx_dim % 8) return "ctx_dim must be a positive multiple of 8";
  if (c.temb_in < 2 || c.temb_in % 8 || c.temb_dim < 8 || c.temb_dim % 8)
    return "temb_in and temb_dim must be multiples of 8";
  if (c.add_in) {
    if (c.add_in != c.pooled_dim + c.n_time_ids * c.time_id_dim) return "add_in must equal pooled + ids*id_dim";
    if (c.add_in % 8 || c.time_id_dim % 2 || c.n_time_ids < 0 || c.n_time_ids > 64 || c.pooled_dim < 0)
      return "unsupported added-embedding shape";
  }
  if (c.max_requests < 1 || c.max_requests > 64) return "max_requests must be in [1, 64]";
  for (int l = 0; l < c.n_levels; ++l) {
    const int ch = c.ch[l];
    if (ch < 8 || ch % 8 || ch % c.gn_groups) return "ch[l] must be multiples of 8 and of gn_groups";
    if (ch > 2048) return "ch[l] must be <= 2048";
    if (c.tx_depth[l] < 0) return "tx_depth must be >= 0";
  }
  if (c.mid_tx_depth < 0) return "mid_tx_depth must be >= 0";
  for (int l = 0; l < c.n_levels; ++l) {
    const bool has_tx = c.tx_depth[l] > 0 || (l == c.n_levels - 1 && c.mid_tx_depth > 0);
    if (!has_tx) continue;
    const int ch = c.ch[l];
    if (c.heads && ch % c.heads) return "ch[l] must be divisible by heads";
    if (c.head_dim && ch % c.head_dim) return "ch[l] must be divisible by head_dim";
    const int d = c.heads ? ch / c.heads : c.head_dim;
    if (d % 8) return "head width must be a multiple of 8";
    if (c.dtype == SD_BF16) {
      if (!attention_width_ok(d)) return "bf16 head width must round up (to 16) to 16..96, 128, 160, 192 or 256";
    } else if (d > 64) {
      return "fp32 head width must be <= 64";
    }
  }
  return "";
}

}  // namespace sd
