#include "net.hpp"

#include "kernels.hpp"

namespace ekya {

Net Net::build(int n_classes, int dt, int hidden) {
  Net n;
  n.n_classes = n_classes;
  n.dt = dt;
  n.hidden = hidden;
  long long off = 0, sh = 0, bnc = 0;
  const int vec = dtype_vec(dt);

  auto add_bn = [&](int C, int stage) {
    BnL b;
    b.C = C;
    b.stage = stage;
    b.g = off;
    b.b = off + C;
    b.rm = off + 2 * C;
    b.rv = off + 3 * C;
    b.st = bnc;
    off += 4LL * C;
    bnc += C;
    n.bn.push_back(b);
    return (int)n.bn.size() - 1;
  };
  auto add_conv = [&](int cin, int cout, int R, int stride, int pad, int stage) {
    ConvL c;
    c.cin = cin;
    c.cout = cout;
    c.R = c.S = R;
    c.stride = stride;
    c.pad = pad;
    c.stage = stage;
    c.off = off;
    off += (long long)cout * cin * R * R;
    c.cin_pad = (cin % vec == 0) ? cin : ((cin + vec - 1) / vec) * vec;
    c.sh_krsc = sh;
    sh += (long long)cout * R * R * c.cin_pad;
    if (stage > 0) {
      c.sh_crsk = sh;
      sh += (long long)cout * R * R * cin;
    } else {
      c.sh_crsk = -1;
    }
    n.conv.push_back(c);
    int ci = (int)n.conv.size() - 1;
    n.conv[ci].bn = add_bn(cout, stage);
    return ci;
  };

  n.stage_begin[0] = 0;
  add_conv(3, 64, 7, 2, 3, 0);
  int cin = 64;
  for (int si = 0; si < 4; ++si) {
    n.stage_begin[si + 1] = off;
    const int w = n.widths[si];
    for (int bi = 0; bi < 2; ++bi) {
      const int stride = (si > 0 && bi == 0) ? 2 : 1;
      BlockL b;
      b.stage = si + 1;
      b.c1 = add_conv(cin, w, 3, stride, 1, si + 1);
      b.c2 = add_conv(w, w, 3, 1, 1, si + 1);
      b.cd = (stride != 1 || cin != w) ? add_conv(cin, w, 1, stride, 0, si + 1) : -1;
      n.blk.push_back(b);
      cin = w;
    }
  }
  n.stage_begin[5] = off;
  if (hidden > 0) {  // fc.0 (hidden x 512), fc.2 (classes x hidden)
    n.fc1_w = off;
    off += (long long)hidden * 512;
    n.fc1_b = off;
    off += hidden;
  }
  n.fc_w = off;
  off += (long long)n_classes * n.head_in();
  n.fc_b = off;
  off += n_classes;
  n.stage_begin[6] = off;
  n.total = off;
  n.bn_channels = bnc;
  n.shadow_elems = sh;
  return n;
}

std::vector<long long> Net::permute_table() const {
  // rows (off, K, C, R, S), sorted by offset; non-conv segments use (off, n, 1, 1, 1)
  std::vector<long long> t;
  long long cur = 0;
  size_t bi = 0;
  for (const ConvL& c : conv) {
    if (c.off > cur) {  // BatchNorm vectors before this conv
      t.insert(t.end(), {cur, c.off - cur, 1, 1, 1});
    }
    t.insert(t.end(), {c.off, c.cout, c.cin, c.R, c.S});
    cur = c.off + (long long)c.cout * c.cin * c.R * c.S;
  }
  (void)bi;
  if (total > cur) t.insert(t.end(), {cur, total - cur, 1, 1, 1});
  return t;
}

std::vector<long long> Net::fold_table(int lo, int hi) const {
  std::vector<long long> t;
  for (const BnL& b : bn)
    if (b.stage >= lo && b.stage <= hi) t.insert(t.end(), {b.g, b.b, b.rm, b.rv, b.C, 2 * b.st});
  return t;
}

std::vector<long long> Net::pack_table(int lo, int hi, bool with_crsk) const {
  std::vector<long long> t;
  for (const ConvL& c : conv)
    if (c.stage >= lo && c.stage <= hi)
      t.insert(t.end(), {c.off, c.cout, c.R, c.S, c.cin, c.cin_pad, c.sh_krsc,
                         with_crsk ? c.sh_crsk : -1LL});
  return t;
}

Geo Geo::build(const Net& net, int H, int W) {
  Geo g;
  g.H = H;
  g.W = W;
  g.ih.resize(net.conv.size());
  g.iw = g.oh = g.ow = g.ih;
  auto o = [](int n, int k, int s, int p) { return (n + 2 * p - k) / s + 1; };
  const ConvL& st = net.conv[0];
  g.ih[0] = H;
  g.iw[0] = W;
  g.sh = g.oh[0] = o(H, st.R, st.stride, st.pad);
  g.sw = g.ow[0] = o(W, st.S, st.stride, st.pad);
  g.mh = (g.sh - 1) / 2 + 1;
  g.mw = (g.sw - 1) / 2 + 1;
  int h = g.mh, w = g.mw;
  for (const BlockL& b : net.blk) {
    for (int ci : {b.c1, b.cd}) {
      if (ci < 0) continue;
      const ConvL& c = net.conv[ci];
      g.ih[ci] = h;
      g.iw[ci] = w;
      g.oh[ci] = o(h, c.R, c.stride, c.pad);
      g.ow[ci] = o(w, c.S, c.stride, c.pad);
    }
    const int h1 = g.oh[b.c1], w1 = g.ow[b.c1];
    g.ih[b.c2] = h1;
    g.iw[b.c2] = w1;
    g.oh[b.c2] = h1;
    g.ow[b.c2] = w1;
    h = h1;
    w = w1;
    g.lh[b.stage] = h;
    g.lw[b.stage] = w;
  }
  return g;
}

int Geo::stage_in_channels(const Net& net, int s) const {
  if (s == 0) return net.conv[0].cin_pad;
  if (s == 1) return 64;
  if (s == 5) return 512;
  return net.widths[s - 2];
}

long long Geo::stage_in_elems(const Net& net, int s) const {
  if (s == 0) return (long long)H * W * net.conv[0].cin_pad;
  if (s == 1) return (long long)mh * mw * 64;
  if (s == 5) return 512;
  return (long long)lh[s - 1] * lw[s - 1] * net.widths[s - 2];
}

}  // namespace ekya
