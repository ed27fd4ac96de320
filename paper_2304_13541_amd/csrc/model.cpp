// Architectures and their executor.
//
// The paper's workloads (Sec. 3, Sec. 6.3, Table model_characteristics)
// are stock image classifiers and a recurrent model.  Each architecture here
// is a flat list of kernel launches over NHWC bf16 activation buffers:
//   tinycnn      4 x (conv3x3 + BN + ReLU), 2x2 max pools after convs 2 and 4,
//                global average pool, FC 64 -> 10
//   resnet50     v1.5 bottlenecks [3,4,6,3] (stride on the 3x3), 7x7/2 stem,
//                3x3/2 max pool, global average pool, FC 2048 -> 1000
//   mobilenetv2  width 1.0 inverted residuals (t,c,n,s) table, ReLU6,
//                linear projections, residual when stride 1 and Cin == Cout
//   vgg19        16 conv3x3 (+bias, ReLU, no BN) in 5 stages, 2x2 max pools,
//                FC 25088 -> 4096 -> 4096 -> 1000 (flattened in (h, w, c) order)
//   lstm2        2-layer LSTM, input 512, hidden 1024, 50 steps
//   bert         BERT-base encoder on 20-token sequences (10-word sentences):
//                embeddings + layer norm, 12 post-norm layers (fused q|k|v
//                projection, 12-head attention, output projection +
//                residual, layer norm, GELU feed-forward 3072 + residual,
//                layer norm), tanh pooler on the first token, 2 classes
//   bert_long    the same on 40-token sequences (20-word sentences)
// Tensor indices follow layer order with weight before bias; BN statistics
// are the constants gamma 1, beta 0, mean 0, var 1, eps 1e-5, folded into a
// per-channel fp32 scale/shift of the producing convolution's epilogue.  The
// transformer's weights and biases are N(0, 0.02^2) (the He rule with fan-in
// 5000) and its layer norms have gain 1, bias 0 and eps 1e-12.
#include "model.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>

namespace dstack {

namespace {

constexpr double BN_EPS = 1e-5;
constexpr size_t SPLITK_WS_BYTES = (size_t)32 << 20;

struct Builder {
  Model& m;
  std::vector<int> free_ids;

  explicit Builder(Model& mm) : m(mm) {}

  int tensor(int64_t numel, int dist, int fan_in, int layout = 0, int d0 = 0, int d1 = 0, int d2 = 0, int d3 = 0) {
    TensorSpec t;
    t.numel = numel;
    t.dist = dist;
    t.fan_in = fan_in;
    t.layout = layout;
    t.d0 = d0; t.d1 = d1; t.d2 = d2; t.d3 = d3;
    t.dev_off = m.n_weights;
    m.n_weights += (dev_numel(t) + 127) / 128 * 128;  // 256-byte aligned tensors
    m.tensors.push_back(t);
    return (int)m.tensors.size() - 1;
  }
  int64_t f32(int64_t n) {
    int64_t off = m.n_fp32;
    m.n_fp32 += (n + 63) / 64 * 64;
    return off;
  }
  int alloc(int64_t elems) {
    if (!free_ids.empty()) {
      int id = free_ids.back();
      free_ids.pop_back();
      m.buf_elems[id] = std::max(m.buf_elems[id], elems);
      return id;
    }
    m.buf_elems.push_back(elems);
    return (int)m.buf_elems.size() - 1;
  }
  void release(int id) {
    if (id >= 0) free_ids.push_back(id);
  }
};

struct Shape {
  int buf, H, W, C;
};

class ArchBuilder {
 public:
  ArchBuilder(Model& m) : b(m), m(m) {}
  Builder b;
  Model& m;

  void push(const Op& op) { m.ops.push_back(op); }

  // conv from tensor wt (logical [K][R][R][Cl]); input shape s (C possibly padded)
  Shape conv(const Shape& s, int wt, int K, int R, int stride, int pad, bool bn, int bias_t, int act, int res_buf,
             int C_true, int out_buf = -100) {
    Op op;
    op.kind = OP_CONV;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.K = K; op.R = R; op.S = R; op.stride = stride; op.pad = pad;
    op.act = act;
    op.Ho = out_dim(s.H, R, stride, pad);
    op.Wo = out_dim(s.W, R, stride, pad);
    op.C_true = C_true;
    op.w_off = m.tensors[wt].dev_off;
    op.res = res_buf;
    if (bn) op.scale_off = b.f32(K);
    if (bn || bias_t >= 0) op.shift_off = b.f32(K);
    op.out = (out_buf == -100) ? b.alloc((int64_t)op.Ho * op.Wo * K) : out_buf;
    op.w_t = wt;
    op.bias_t = bias_t;
    op.bn = bn ? 1 : 0;
    push(op);
    return Shape{op.out, op.Ho, op.Wo, K};
  }
  // stem conv straight from the 3-channel input image (weights [K][R][R][4])
  Shape conv_rgb(int H, int W, int wt, int K, int R, int stride, int pad, bool bn, int bias_t, int act) {
    Op op;
    op.kind = OP_CONV_RGB;
    op.in = BUF_IN;
    op.H = H; op.W = W; op.C = 3; op.K = K; op.R = R; op.S = R; op.stride = stride; op.pad = pad;
    op.act = act;
    op.Ho = out_dim(H, R, stride, pad);
    op.Wo = out_dim(W, R, stride, pad);
    op.C_true = 3;
    op.w_off = m.tensors[wt].dev_off;
    op.scale_off = b.f32(K);  // 1 without BN
    op.shift_off = b.f32(K);
    op.out = b.alloc((int64_t)op.Ho * op.Wo * K);
    op.w_t = wt;
    op.bias_t = bias_t;
    op.bn = bn ? 1 : 0;
    push(op);
    return Shape{op.out, op.Ho, op.Wo, K};
  }
  // expand 1x1 conv + BN + ReLU6 and depthwise 3x3 + BN + ReLU6 in one kernel
  Shape expand_dw(const Shape& s, int we, int Ce, int wd, int stride) {
    Op op;
    op.kind = OP_EXPAND_DW;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.K = Ce; op.R = 3; op.S = 3; op.stride = stride; op.pad = 1;
    op.act = ACT_RELU6;
    op.act2 = ACT_RELU6;
    op.Ho = out_dim(s.H, 3, stride, 1);
    op.Wo = out_dim(s.W, 3, stride, 1);
    op.C_true = s.C;
    op.w_off = m.tensors[we].dev_off;
    op.w2_off = m.tensors[wd].dev_off;
    op.scale_off = b.f32(Ce);
    op.shift_off = b.f32(Ce);
    op.scale2_off = b.f32(Ce);
    op.shift2_off = b.f32(Ce);
    op.out = b.alloc((int64_t)op.Ho * op.Wo * Ce);
    op.w_t = we;
    op.bn = 1;
    push(op);
    return Shape{op.out, op.Ho, op.Wo, Ce};
  }
  Shape dw(const Shape& s, int wt, int stride) {
    Op op;
    op.kind = OP_DW;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.K = s.C; op.R = 3; op.S = 3; op.stride = stride; op.pad = 1;
    op.act = ACT_RELU6;
    op.Ho = out_dim(s.H, 3, stride, 1);
    op.Wo = out_dim(s.W, 3, stride, 1);
    op.C_true = s.C;
    op.w_off = m.tensors[wt].dev_off;
    op.scale_off = b.f32(s.C);
    op.shift_off = b.f32(s.C);
    op.out = b.alloc((int64_t)op.Ho * op.Wo * s.C);
    op.w_t = wt;
    op.bn = 1;
    push(op);
    return Shape{op.out, op.Ho, op.Wo, s.C};
  }
  Shape maxpool(const Shape& s, int k, int stride, int pad) {
    Op op;
    op.kind = OP_MAXPOOL;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.K = s.C; op.R = k; op.S = k; op.stride = stride; op.pad = pad;
    op.Ho = out_dim(s.H, k, stride, pad);
    op.Wo = out_dim(s.W, k, stride, pad);
    op.out = b.alloc((int64_t)op.Ho * op.Wo * s.C);
    push(op);
    return Shape{op.out, op.Ho, op.Wo, s.C};
  }
  Shape avgpool(const Shape& s) {
    Op op;
    op.kind = OP_AVGPOOL;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.K = s.C;
    op.Ho = 1; op.Wo = 1;
    op.out = b.alloc(s.C);
    push(op);
    return Shape{op.out, 1, 1, s.C};
  }
  // token ids -> word + position + type embedding -> layer norm, [T][H] per item
  Shape embed_ln(int T, int vocab, int H, int we, int pe, int te) {
    Op op;
    op.kind = OP_EMBED_LN;
    op.in = BUF_IN;
    op.T = T; op.C = H; op.K = vocab;
    op.H = 1; op.W = T; op.Ho = 1; op.Wo = T;
    op.w_off = m.tensors[we].dev_off;
    op.w2_off = m.tensors[pe].dev_off;
    op.w3_off = m.tensors[te].dev_off;
    op.out = b.alloc((int64_t)T * H);
    push(op);
    return Shape{op.out, 1, T, H};
  }
  Shape layernorm(const Shape& s) {
    Op op;
    op.kind = OP_LAYERNORM;
    op.in = s.buf;
    op.H = s.H; op.W = s.W; op.C = s.C; op.Ho = s.H; op.Wo = s.W;
    op.out = b.alloc((int64_t)s.H * s.W * s.C);
    push(op);
    return Shape{op.out, s.H, s.W, s.C};
  }
  // fused q|k|v [T][3*width] -> attention output [T][width]
  Shape attention(const Shape& s, int heads) {
    Op op;
    op.kind = OP_ATTENTION;
    op.in = s.buf;
    op.T = s.W; op.C = s.C / 3; op.K = heads;
    op.H = 1; op.W = s.W; op.Ho = 1; op.Wo = s.W;
    op.out = b.alloc((int64_t)s.W * (s.C / 3));
    push(op);
    return Shape{op.out, 1, s.W, s.C / 3};
  }
  Shape fc(const Shape& s, int wt, int bt, int O, int act, bool last) {
    Op op;
    op.kind = OP_FC;
    op.in = s.buf;
    op.C = s.H * s.W * s.C;  // flattened (h, w, c)
    op.K = O;
    op.act = act;
    op.w_off = m.tensors[wt].dev_off;
    op.shift_off = b.f32(O);
    op.out_f32 = last ? 1 : 0;
    op.out = last ? BUF_OUT : b.alloc(O);
    op.w_t = wt;
    op.bias_t = bt;
    push(op);
    return Shape{op.out, 1, 1, O};
  }
  void done(const Shape& s, const Shape& keep) {
    if (s.buf != keep.buf) b.release(s.buf);
  }
};

void build_tiny(ArchBuilder& A) {
  Model& m = A.m;
  m.in_h = m.in_w = 32;
  m.in_c = 3;
  m.out_features = 10;
  const int ch[5] = {3, 16, 32, 32, 64};
  int wt[4];
  for (int l = 0; l < 4; ++l)
    wt[l] = A.b.tensor((int64_t)ch[l + 1] * 9 * ch[l], DIST_HE, 9 * ch[l], l == 0 ? 3 : 0, ch[l + 1], 3, 3, ch[l]);
  int fw = A.b.tensor(640, DIST_HE, 64);
  int fb = A.b.tensor(10, DIST_ZERO, 0);
  Shape x = A.conv_rgb(32, 32, wt[0], ch[1], 3, 1, 1, true, -1, ACT_RELU);
  for (int l = 1; l < 4; ++l) {
    Shape y = A.conv(x, wt[l], ch[l + 1], 3, 1, 1, true, -1, ACT_RELU, BUF_NONE, ch[l]);
    A.b.release(x.buf);
    x = y;
    if (l == 1 || l == 3) {
      Shape p = A.maxpool(x, 2, 2, 0);
      A.b.release(x.buf);
      x = p;
    }
  }
  Shape g = A.avgpool(x);
  A.b.release(x.buf);
  A.fc(g, fw, fb, 10, ACT_NONE, true);
}

void build_r50(ArchBuilder& A) {
  Model& m = A.m;
  m.in_h = m.in_w = 224;
  m.in_c = 3;
  m.out_features = 1000;
  static const int stages[4][3] = {{3, 64, 1}, {4, 128, 2}, {6, 256, 2}, {3, 512, 2}};
  int stem = A.b.tensor(64L * 49 * 3, DIST_HE, 147, 3, 64, 7, 7, 3);
  struct Blk {
    int w1, w2, w3, wd, planes, stride, cin;
  };
  std::vector<Blk> blks;
  int cin = 64;
  for (int st = 0; st < 4; ++st) {
    int planes = stages[st][1];
    for (int i = 0; i < stages[st][0]; ++i) {
      Blk k;
      k.planes = planes;
      k.stride = i == 0 ? stages[st][2] : 1;
      k.cin = cin;
      k.w1 = A.b.tensor((int64_t)planes * cin, DIST_HE, cin, 0, planes, 1, 1, cin);
      k.w2 = A.b.tensor((int64_t)planes * 9 * planes, DIST_HE, 9 * planes, 0, planes, 3, 3, planes);
      k.w3 = A.b.tensor((int64_t)4 * planes * planes, DIST_HE, planes, 0, 4 * planes, 1, 1, planes);
      k.wd = i == 0 ? A.b.tensor((int64_t)4 * planes * cin, DIST_HE, cin, 0, 4 * planes, 1, 1, cin) : -1;
      blks.push_back(k);
      cin = 4 * planes;
    }
  }
  int fw = A.b.tensor(1000L * 2048, DIST_HE, 2048);
  int fb = A.b.tensor(1000, DIST_ZERO, 0);

  Shape s = A.conv_rgb(224, 224, stem, 64, 7, 2, 3, true, -1, ACT_RELU);
  Shape cur = A.maxpool(s, 3, 2, 1);
  A.b.release(s.buf);
  for (const Blk& k : blks) {
    Shape t1 = A.conv(cur, k.w1, k.planes, 1, 1, 0, true, -1, ACT_RELU, BUF_NONE, k.cin);
    Shape t2 = A.conv(t1, k.w2, k.planes, 3, k.stride, 1, true, -1, ACT_RELU, BUF_NONE, k.planes);
    A.b.release(t1.buf);
    Shape sc = cur;
    if (k.wd >= 0) sc = A.conv(cur, k.wd, 4 * k.planes, 1, k.stride, 0, true, -1, ACT_NONE, BUF_NONE, k.cin);
    Shape out = A.conv(t2, k.w3, 4 * k.planes, 1, 1, 0, true, -1, ACT_RELU, sc.buf, k.planes);
    A.b.release(t2.buf);
    if (sc.buf != cur.buf) A.b.release(sc.buf);
    A.b.release(cur.buf);
    cur = out;
  }
  Shape g = A.avgpool(cur);
  A.b.release(cur.buf);
  A.fc(g, fw, fb, 1000, ACT_NONE, true);
}

void build_mbv2(ArchBuilder& A) {
  Model& m = A.m;
  m.in_h = m.in_w = 224;
  m.in_c = 3;
  m.out_features = 1000;
  static const int cfg[7][4] = {{1, 16, 1, 1}, {6, 24, 2, 2}, {6, 32, 3, 2}, {6, 64, 4, 2},
                                {6, 96, 3, 1}, {6, 160, 3, 2}, {6, 320, 1, 1}};
  int stem = A.b.tensor(32L * 9 * 3, DIST_HE, 27, 3, 32, 3, 3, 3);
  struct Blk {
    int we, wd, wp, cin, hid, cout, stride;
  };
  std::vector<Blk> blks;
  int cin = 32;
  for (int g = 0; g < 7; ++g) {
    int t = cfg[g][0], c = cfg[g][1], n = cfg[g][2], s = cfg[g][3];
    for (int i = 0; i < n; ++i) {
      Blk k;
      k.cin = cin;
      k.hid = cin * t;
      k.cout = c;
      k.stride = i == 0 ? s : 1;
      k.we = t != 1 ? A.b.tensor((int64_t)k.hid * cin, DIST_HE, cin, 0, k.hid, 1, 1, cin) : -1;
      k.wd = A.b.tensor((int64_t)k.hid * 9, DIST_HE, 9, 2, k.hid, 3, 3, 1);
      k.wp = A.b.tensor((int64_t)c * k.hid, DIST_HE, k.hid, 0, c, 1, 1, k.hid);
      blks.push_back(k);
      cin = c;
    }
  }
  int wl = A.b.tensor(1280L * 320, DIST_HE, 320, 0, 1280, 1, 1, 320);
  int fw = A.b.tensor(1000L * 1280, DIST_HE, 1280);
  int fb = A.b.tensor(1000, DIST_ZERO, 0);

  Shape cur = A.conv_rgb(224, 224, stem, 32, 3, 2, 1, true, -1, ACT_RELU6);
  for (const Blk& k : blks) {
    Shape d;
    if (k.we >= 0 && k.cin % 8 == 0 && k.cin <= 160 && k.hid % 48 == 0) {
      d = A.expand_dw(cur, k.we, k.hid, k.wd, k.stride);
    } else {
      Shape e = cur;
      if (k.we >= 0) e = A.conv(cur, k.we, k.hid, 1, 1, 0, true, -1, ACT_RELU6, BUF_NONE, k.cin);
      d = A.dw(e, k.wd, k.stride);
      if (e.buf != cur.buf) A.b.release(e.buf);
    }
    bool res = k.stride == 1 && k.cin == k.cout;
    Shape p = A.conv(d, k.wp, k.cout, 1, 1, 0, true, -1, ACT_NONE, res ? cur.buf : BUF_NONE, k.hid);
    A.b.release(d.buf);
    A.b.release(cur.buf);
    cur = p;
  }
  Shape l = A.conv(cur, wl, 1280, 1, 1, 0, true, -1, ACT_RELU6, BUF_NONE, 320);
  A.b.release(cur.buf);
  Shape g = A.avgpool(l);
  A.b.release(l.buf);
  A.fc(g, fw, fb, 1000, ACT_NONE, true);
}

void build_vgg(ArchBuilder& A) {
  Model& m = A.m;
  m.in_h = m.in_w = 224;
  m.in_c = 3;
  m.out_features = 1000;
  static const int nconv[5] = {2, 2, 4, 4, 4};
  static const int chs[5] = {64, 128, 256, 512, 512};
  std::vector<int> wts, bts, couts, cins;
  int cin = 3;
  for (int st = 0; st < 5; ++st)
    for (int i = 0; i < nconv[st]; ++i) {
      int cout = chs[st];
      wts.push_back(A.b.tensor((int64_t)cout * 9 * cin, DIST_HE, 9 * cin, cin == 3 ? 3 : 0, cout, 3, 3, cin));
      bts.push_back(A.b.tensor(cout, DIST_ZERO, 0));
      couts.push_back(cout);
      cins.push_back(cin);
      cin = cout;
    }
  int f1 = A.b.tensor(4096L * 25088, DIST_HE, 25088), b1 = A.b.tensor(4096, DIST_ZERO, 0);
  int f2 = A.b.tensor(4096L * 4096, DIST_HE, 4096), b2 = A.b.tensor(4096, DIST_ZERO, 0);
  int f3 = A.b.tensor(1000L * 4096, DIST_HE, 4096), b3 = A.b.tensor(1000, DIST_ZERO, 0);

  Shape cur = A.conv_rgb(224, 224, wts[0], couts[0], 3, 1, 1, false, bts[0], ACT_RELU);
  size_t li = 1;
  for (int st = 0; st < 5; ++st) {
    for (int i = st == 0 ? 1 : 0; i < nconv[st]; ++i, ++li) {
      Shape y = A.conv(cur, wts[li], couts[li], 3, 1, 1, false, bts[li], ACT_RELU, BUF_NONE, cins[li]);
      A.b.release(cur.buf);
      cur = y;
    }
    Shape p = A.maxpool(cur, 2, 2, 0);
    A.b.release(cur.buf);
    cur = p;
  }
  Shape h1 = A.fc(cur, f1, b1, 4096, ACT_RELU, false);
  A.b.release(cur.buf);
  Shape h2 = A.fc(h1, f2, b2, 4096, ACT_RELU, false);
  A.b.release(h1.buf);
  A.fc(h2, f3, b3, 1000, ACT_NONE, true);
  A.b.release(h2.buf);
}

void build_lstm(ArchBuilder& A) {
  Model& m = A.m;
  m.is_lstm = 1;
  m.seq_len = 50;
  m.in_features = 512;
  m.out_features = 1024;
  m.lstm_T = 50;
  m.lstm_H = 1024;
  int in = 512;
  for (int l = 0; l < 2; ++l) {
    Op op;
    op.kind = OP_LSTM;
    op.T = 50;
    op.I = in;
    op.Hd = 1024;
    op.wih_t = A.b.tensor(4096L * in, DIST_LSTM, 0, 0, 4096, in, 1, 1);
    op.whh_t = A.b.tensor(4096L * 1024, DIST_LSTM, 0, 0, 4096, 1024, 1, 1);
    op.bih_t = A.b.tensor(4096, DIST_LSTM, 0);
    op.bhh_t = A.b.tensor(4096, DIST_LSTM, 0);
    op.wih_off = m.tensors[op.wih_t].dev_off;
    op.whh_off = m.tensors[op.whh_t].dev_off;
    op.bias_off = A.b.f32(4096);
    // layer 1 reads the model input and keeps its bf16 h in the workspace;
    // layer 2 reads that h and writes the fp32 output
    op.in = l == 0 ? BUF_IN : BUF_NONE;
    op.out = l == 0 ? BUF_NONE : BUF_OUT;
    A.push(op);
    in = 1024;
  }
}

void build_bert(ArchBuilder& A, int T) {
  Model& m = A.m;
  const int H = 768, heads = 12, FF = 3072, vocab = 30522, L = 12, FAN = 5000;
  m.input_tokens = 1;
  m.seq_len = T;
  m.out_features = 2;
  int we = A.b.tensor((int64_t)vocab * H, DIST_HE, FAN);
  int pe = A.b.tensor(512L * H, DIST_HE, FAN);
  int te = A.b.tensor(2L * H, DIST_HE, FAN);
  std::vector<int> t;
  for (int l = 0; l < L; ++l) {
    t.push_back(A.b.tensor(3L * H * H, DIST_HE, FAN));
    t.push_back(A.b.tensor(3L * H, DIST_HE, FAN));
    t.push_back(A.b.tensor((int64_t)H * H, DIST_HE, FAN));
    t.push_back(A.b.tensor(H, DIST_HE, FAN));
    t.push_back(A.b.tensor((int64_t)FF * H, DIST_HE, FAN));
    t.push_back(A.b.tensor(FF, DIST_HE, FAN));
    t.push_back(A.b.tensor((int64_t)H * FF, DIST_HE, FAN));
    t.push_back(A.b.tensor(H, DIST_HE, FAN));
  }
  int wp = A.b.tensor((int64_t)H * H, DIST_HE, FAN), bp = A.b.tensor(H, DIST_HE, FAN);
  int wc = A.b.tensor(2L * H, DIST_HE, FAN), bc = A.b.tensor(2, DIST_HE, FAN);

  Shape x = A.embed_ln(T, vocab, H, we, pe, te);
  for (int l = 0; l < L; ++l) {
    const int* w = &t[8 * l];
    Shape qkv = A.conv(x, w[0], 3 * H, 1, 1, 0, false, w[1], ACT_NONE, BUF_NONE, H);
    Shape att = A.attention(qkv, heads);
    A.b.release(qkv.buf);
    Shape a = A.conv(att, w[2], H, 1, 1, 0, false, w[3], ACT_NONE, x.buf, H);  // + residual x
    A.b.release(att.buf);
    A.b.release(x.buf);
    Shape a1 = A.layernorm(a);
    A.b.release(a.buf);
    Shape f = A.conv(a1, w[4], FF, 1, 1, 0, false, w[5], ACT_GELU, BUF_NONE, H);
    Shape g = A.conv(f, w[6], H, 1, 1, 0, false, w[7], ACT_NONE, a1.buf, FF);  // + residual a1
    A.b.release(f.buf);
    A.b.release(a1.buf);
    x = A.layernorm(g);
    A.b.release(g.buf);
  }
  // pooler on the first token of each sequence: a 1x1 convolution of stride T over the row of T tokens
  Shape p = A.conv(x, wp, H, 1, T, 0, false, bp, ACT_TANH, BUF_NONE, H);
  A.b.release(x.buf);
  A.fc(p, wc, bc, 2, ACT_NONE, true);
  A.b.release(p.buf);
}

}  // namespace

dstack_status build_arch(const std::string& arch, Model& m) {
  m.arch = arch;
  ArchBuilder A(m);
  if (arch == "tinycnn")
    build_tiny(A);
  else if (arch == "resnet50")
    build_r50(A);
  else if (arch == "mobilenetv2")
    build_mbv2(A);
  else if (arch == "vgg19")
    build_vgg(A);
  else if (arch == "lstm2")
    build_lstm(A);
  else if (arch == "bert")
    build_bert(A, 20);
  else if (arch == "bert_long")
    build_bert(A, 40);
  else
    return fail(DSTACK_E_UNSUPPORTED, "unknown arch '" + arch + "'");
  return DSTACK_OK;
}

static double bf16_bits_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return (double)f;
}

dstack_status upload_weights(Model& m) {
  std::vector<uint16_t> arena((size_t)m.n_weights, 0);
  std::vector<std::vector<uint16_t>> logical(m.tensors.size());
  for (size_t i = 0; i < m.tensors.size(); ++i) {
    const TensorSpec& t = m.tensors[i];
    std::vector<uint16_t> v((size_t)t.numel);
    generate_tensor(m.seed, (int)i, t, v.data());
    uint16_t* dst = arena.data() + t.dev_off;
    if (t.layout == 0) {
      std::memcpy(dst, v.data(), v.size() * 2);
    } else if (t.layout == 1) {  // [K][R][S][C] -> [K][R][S][8]
      int64_t krs = (int64_t)t.d0 * t.d1 * t.d2;
      for (int64_t q = 0; q < krs; ++q)
        for (int c = 0; c < t.d3; ++c) dst[q * 8 + c] = v[(size_t)(q * t.d3 + c)];
    } else if (t.layout == 3) {  // RGB stem [K][R][S][3] -> [K][R][S][4]
      int64_t krs = (int64_t)t.d0 * t.d1 * t.d2;
      for (int64_t q = 0; q < krs; ++q)
        for (int c = 0; c < t.d3; ++c) dst[q * 4 + c] = v[(size_t)(q * t.d3 + c)];
    } else {  // depthwise [C][3][3] -> [3][3][C]
      int C = t.d0;
      for (int c = 0; c < C; ++c)
        for (int rs = 0; rs < 9; ++rs) dst[(size_t)rs * C + c] = v[(size_t)c * 9 + rs];
    }
    // keep small tensors (biases) for folding
    if (t.numel <= 8192) logical[i] = std::move(v);
  }
  m.fp32_host.assign((size_t)m.n_fp32, 0.f);
  const double bn_scale = 1.0 / std::sqrt(1.0 + BN_EPS);  // gamma / sqrt(var + eps) with gamma 1, var 1
  for (size_t o = 0; o < m.ops.size(); ++o) {
    const Op& op = m.ops[o];
    const Op& ex = op;
    if (op.kind == OP_LSTM) {
      const auto& bi = logical[ex.bih_t];
      const auto& bh = logical[ex.bhh_t];
      for (int j = 0; j < 4 * op.Hd; ++j)
        m.fp32_host[op.bias_off + j] = (float)(bf16_bits_to_double(bi[j]) + bf16_bits_to_double(bh[j]));
      continue;
    }
    int K = op.K;
    for (int k = 0; k < K; ++k) {
      double bias = ex.bias_t >= 0 ? bf16_bits_to_double(logical[ex.bias_t][k]) : 0.0;
      double sc = ex.bn ? bn_scale : 1.0;
      // BN(y + bias) = sc * y + (bias * sc + beta - mean * sc), beta = mean = 0
      if (op.scale_off >= 0) m.fp32_host[op.scale_off + k] = (float)sc;
      if (op.shift_off >= 0) m.fp32_host[op.shift_off + k] = (float)(bias * sc);
      // the fused depthwise stage: BN, no bias
      if (op.scale2_off >= 0) m.fp32_host[op.scale2_off + k] = (float)bn_scale;
      if (op.shift2_off >= 0) m.fp32_host[op.shift2_off + k] = 0.0f;
    }
  }
  DS_HIP(hipMalloc(&m.d_w, (size_t)m.n_weights * 2));
  DS_HIP(hipMemcpy(m.d_w, arena.data(), (size_t)m.n_weights * 2, hipMemcpyHostToDevice));
  // The weight-streaming operands again, in the MFMA fragment order their
  // kernels read (16 rows x 32 deep per 1 KB block, zero past the matrix):
  // FC weights [O][I] with row tile ot = rows 16 ot .. 16 ot + 15; LSTM W_hh
  // [4H][H] with row tile rt = the rows (gate, unit) = (r / 4, 4 rt + r % 4).
  auto pack = [](const uint16_t* src, int rows, int cols, int tiles, auto row_of, uint16_t* dst) {
    const int nks = (cols + 31) / 32;
    for (int t = 0; t < tiles; ++t)
      for (int st = 0; st < nks; ++st)
        for (int r = 0; r < 16; ++r) {
          const int row = row_of(t, r);
          uint16_t* d = dst + (((size_t)t * nks + st) * 16 + r) * 32;
          for (int kk = 0; kk < 32; ++kk) {
            const int k = st * 32 + kk;
            d[kk] = row < rows && k < cols ? src[(size_t)row * cols + k] : 0;
          }
        }
  };
  m.n_wp = 0;
  for (Op& op : m.ops) {
    op.wp_off = -1;
    if (op.kind == OP_FC) {
      op.wp_off = m.n_wp;
      m.n_wp += ((int64_t)(op.K + 15) / 16 * 16 * ((op.C + 31) / 32 * 32) + 127) / 128 * 128;
    } else if (op.kind == OP_LSTM) {
      op.wp_off = m.n_wp;
      m.n_wp += ((int64_t)4 * op.Hd * op.Hd + 127) / 128 * 128;
    }
  }
  if (m.n_wp > 0) {
    std::vector<uint16_t> packed((size_t)m.n_wp, 0);
    for (const Op& op : m.ops) {
      if (op.kind == OP_FC)
        pack(arena.data() + op.w_off, op.K, op.C, (op.K + 15) / 16, [](int t, int r) { return 16 * t + r; },
             packed.data() + op.wp_off);
      else if (op.kind == OP_LSTM)
        pack(arena.data() + op.whh_off, 4 * op.Hd, op.Hd, op.Hd / 4,
             [H = op.Hd](int t, int r) { return (r >> 2) * H + 4 * t + (r & 3); }, packed.data() + op.wp_off);
    }
    DS_HIP(hipMalloc(&m.d_wp, (size_t)m.n_wp * 2));
    DS_HIP(hipMemcpy(m.d_wp, packed.data(), (size_t)m.n_wp * 2, hipMemcpyHostToDevice));
  }
  if (m.n_fp32 > 0) {
    DS_HIP(hipMalloc(&m.d_f32, (size_t)m.n_fp32 * 4));
    DS_HIP(hipMemcpy(m.d_f32, m.fp32_host.data(), (size_t)m.n_fp32 * 4, hipMemcpyHostToDevice));
  }
  return DSTACK_OK;
}

Workspace::~Workspace() {
  for (auto& kv : graphs) (void)hipGraphExecDestroy(kv.second);
}

Model::~Model() {
  for (auto& kv : ws)
    if (kv.second->base) (void)hipFree(kv.second->base);
  if (d_w) (void)hipFree(d_w);
  if (d_f32) (void)hipFree(d_f32);
  if (d_wp) (void)hipFree(d_wp);
  if (sweep_in) (void)hipFree(sweep_in);
  if (sweep_out) (void)hipFree(sweep_out);
}

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

void release_workspace(Model& m, int pid) {
  std::lock_guard<std::mutex> g(m.ws_mu);
  auto it = m.ws.find(pid);
  if (it == m.ws.end() || it->second->busy.load()) return;
  void* base = it->second->base;
  m.ws.erase(it);  // destroys its graph execs
  if (base) (void)hipFree(base);
}

dstack_status get_workspace(Model& m, int pid, int n_cu, hipStream_t st, Workspace** out) {
  std::lock_guard<std::mutex> g(m.ws_mu);
  auto it = m.ws.find(pid);
  if (it != m.ws.end()) {
    *out = it->second.get();
    return DSTACK_OK;
  }
  auto w = std::make_unique<Workspace>();
  std::vector<size_t> offs;
  size_t total = 0;
  for (int64_t e : m.buf_elems) {
    offs.push_back(total);
    total += align256((size_t)e * m.max_batch * 2);
  }
  // split-K partial sums: a conv split plan stops doubling once splits *
  // tiles reaches 2 * n_cu (so stays below 4 * 256 tiles of at most 128 x 64
  // fp32 values = 32 MB), an FC split needs at most 16 * 32 * O fp32 values;
  // a shape asking for more runs with fewer splits
  size_t sk = 0;
  for (const Op& op : m.ops)
    if (op.kind == OP_CONV || op.kind == OP_FC) sk = SPLITK_WS_BYTES;
  size_t sk_off = total;
  total += align256(sk);
  const size_t cnt_off = total;
  if (sk) total += align256(SPLITK_TILE_COUNTERS * sizeof(unsigned));
  size_t gx_off = 0, c_off = 0, h0_off = 0, h1_off = 0, hp_off = 0;
  if (m.is_lstm) {
    gx_off = total;
    total += align256((size_t)m.lstm_T * m.max_batch * 4 * m.lstm_H * 4);
    c_off = total;
    total += align256((size_t)m.max_batch * m.lstm_H * 4);
    h0_off = total;
    total += align256((size_t)m.lstm_T * m.max_batch * m.lstm_H * 2);
    h1_off = total;
    total += align256((size_t)m.lstm_T * m.max_batch * m.lstm_H * 2);
    hp_off = total;
    total += align256((size_t)2 * m.max_batch * m.lstm_H * 2);
  }
  DS_HIP(hipMalloc(&w->base, total));
  w->bytes = total;
  char* base = (char*)w->base;
  for (size_t o : offs) w->bufs.push_back(base + o);
  if (sk) {
    w->splitk = (float*)(base + sk_off);
    w->splitk_bytes = sk;
    // the counters start at zero; each fused split-K launch leaves them so
    w->tile_counters = (unsigned*)(base + cnt_off);
    dstack_status zs = DSTACK_OK;
    if (hipMemsetAsync(w->tile_counters, 0, SPLITK_TILE_COUNTERS * sizeof(unsigned), st) != hipSuccess ||
        hipStreamSynchronize(st) != hipSuccess)
      zs = fail(DSTACK_E_HIP, "workspace: clearing the split-K counters failed");
    if (zs != DSTACK_OK) {
      (void)hipFree(w->base);
      return zs;
    }
  }
  if (m.is_lstm) {
    w->lstm_gx = (float*)(base + gx_off);
    w->lstm_c = (float*)(base + c_off);
    w->lstm_h[0] = (bf16*)(base + h0_off);
    w->lstm_h[1] = (bf16*)(base + h1_off);
    w->lstm_hp = (bf16*)(base + hp_off);
  }
  *out = w.get();
  m.ws[pid] = std::move(w);
  (void)n_cu;
  return DSTACK_OK;
}

std::vector<LaunchShape>*& shape_recorder() {
  static thread_local std::vector<LaunchShape>* rec = nullptr;
  return rec;
}

void KernelTimer::before() {
  if (dry) {
    unit_l0 = shape_recorder() ? shape_recorder()->size() : 0;
    return;
  }
  if (!pending) {
    (void)hipEventCreate(&pending);
    (void)hipEventRecord(pending, st);
  }
}

DispatchEvents& dispatch_events() {
  static thread_local DispatchEvents ev;
  return ev;
}

void KernelTimer::before_dispatch() {
  if (dry) {
    before();
    return;
  }
  (void)hipEventCreate(&ds_start);
  (void)hipEventCreate(&ds_stop);
  dispatch_events() = DispatchEvents{ds_start, ds_stop};
}

void KernelTimer::after(int kind, double flops, double bytes, int m, int n, int k) {
  if (dry) {
    units.push_back(Unit{kind, unit_l0, shape_recorder() ? shape_recorder()->size() : unit_l0, flops, bytes});
    return;
  }
  if (ds_start) {  // timed by the kernels' own dispatch packets
    recs.push_back(Rec{kind, flops, bytes, ds_start, ds_stop, m, n, k});
    ds_start = ds_stop = nullptr;
    dispatch_events() = DispatchEvents{};
    return;
  }
  hipEvent_t e;
  (void)hipEventCreate(&e);
  (void)hipEventRecord(e, st);
  recs.push_back(Rec{kind, flops, bytes, pending, e, m, n, k});
  pending = nullptr;
}

KernelTimer::~KernelTimer() {
  for (auto& r : recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  if (pending) (void)hipEventDestroy(pending);
  if (ds_start) (void)hipEventDestroy(ds_start);
  if (ds_stop) (void)hipEventDestroy(ds_stop);
  dispatch_events() = DispatchEvents{};
}

static double conv_flops(const Op& op, int b) {
  return 2.0 * b * op.Ho * op.Wo * (double)op.K * op.R * op.S * op.C_true;
}
static double conv_bytes(const Op& op, int b) {
  double in = (double)b * op.H * op.W * op.C_true * 2;
  double w = (double)op.K * op.R * op.S * op.C_true * 2;
  double out = (double)b * op.Ho * op.Wo * op.K * 2;
  return in + w + out * (op.res != BUF_NONE ? 2 : 1);
}

dstack_status lstm_layer_run(const bf16* x, int T, int B, int I, int H, const bf16* w_ih, const bf16* w_hh,
                             const bf16* whh_packed, const float* bias, bf16* h_bf16, float* h_f32, float* gx,
                             float* c, bf16* wp_scratch, bf16* hp, int n_cu, hipStream_t st, KernelTimer* timer) {
  // input projection of all steps at once: gx[t*B + b][:] = W_ih x + b_ih + b_hh (fp32)
  if (timer) timer->before();
  dstack_status s = launch_conv2d_ws(x, T * B, 1, 1, I, w_ih, 4 * H, 1, 1, 1, 0, nullptr, bias, nullptr, ACT_NONE,
                                     gx, true, n_cu, nullptr, 0, nullptr, st);
  if (s != DSTACK_OK) return s;
  if (timer)
    timer->after(KC_MFMA, 2.0 * T * B * I * 4.0 * H,
                 (double)T * B * I * 2 + 4.0 * H * I * 2 + (double)T * B * 4 * H * 4, T * B, 4 * H, I);
  // W_hh in the fragment order of the recurrent product
  const bf16* wp = whh_packed;
  if (!wp) {
    if (timer) timer->before();
    s = launch_lstm_pack_whh(w_hh, wp_scratch, H, st);
    if (s != DSTACK_OK) return s;
    if (timer) timer->after(KC_GLUE, 0.0, 2.0 * 4.0 * H * H * 2, 0, 0, 0);
    wp = wp_scratch;
  }
  for (int t = 0; t < T; ++t) {
    if (timer) timer->before();
    bf16* hp_t = hp + (size_t)(t & 1) * B * H;
    const bf16* hp_prev = hp + (size_t)((t + 1) & 1) * B * H;
    s = launch_lstm_step(gx + (size_t)t * B * 4 * H, wp, t ? hp_prev : nullptr, c, h_bf16 + (size_t)t * B * H, hp_t,
                         h_f32 ? h_f32 + (size_t)t * B * H : nullptr, B, H, t == 0, n_cu, st);
    if (s != DSTACK_OK) return s;
    if (timer)
      timer->after(KC_LSTM, 2.0 * B * H * 4.0 * H,
                   4.0 * H * H * 2 + (double)B * H * 2 + (double)B * 4 * H * 4 + 2.0 * B * H * 4 + 2.0 * B * H * 2 +
                       (h_f32 ? (double)B * H * 4 : 0.0),
                   B, 4 * H, H);
  }
  return DSTACK_OK;
}

dstack_status forward(Model& m, int batch, const void* d_in, void* d_out, Workspace& ws, int n_cu, hipStream_t st,
                      KernelTimer* timer, int n_ops, void** last_out) {
  auto bufp = [&](int id, const void* in, void* out) -> void* {
    if (id == BUF_IN) return const_cast<void*>(in);
    if (id == BUF_OUT) return out;
    if (id == BUF_NONE) return nullptr;
    return ws.bufs[id];
  };
  const float* f32 = m.d_f32;
  const size_t n_run = n_ops < 0 ? m.ops.size() : std::min(m.ops.size(), (size_t)n_ops);
  for (size_t oi = 0; oi < n_run; ++oi) {
    const Op& op = m.ops[oi];
    dstack_status s = DSTACK_OK;
    const bf16* src = (const bf16*)bufp(op.in, d_in, d_out);
    void* dst = bufp(op.out, d_in, d_out);
    if (last_out) *last_out = dst;
    if (op.kind == OP_LSTM) {
      // layer 1 (reads the model input) -> lstm_h[0]; layer 2 -> lstm_h[1] and d_out
      const bf16* x = op.in == BUF_IN ? (const bf16*)d_in : ws.lstm_h[0];
      bf16* hb = op.in == BUF_IN ? ws.lstm_h[0] : ws.lstm_h[1];
      float* hf = op.out == BUF_OUT ? (float*)d_out : nullptr;
      s = lstm_layer_run(x, op.T, batch, op.I, op.Hd, m.d_w + op.wih_off, m.d_w + op.whh_off, m.d_wp + op.wp_off,
                         f32 + op.bias_off, hb, hf, ws.lstm_gx, ws.lstm_c, nullptr, ws.lstm_hp, n_cu, st, timer);
      if (s != DSTACK_OK) return s;
      continue;
    }
    if (timer) {  // convolutions: timestamps of their own dispatches; others: events around them
      if (op.kind == OP_CONV)
        timer->before_dispatch();
      else
        timer->before();
    }
    int kind = KC_GLUE;
    double fl = 0, by = 0;
    int gm = 0, gn = 0, gk = 0;
    switch (op.kind) {
      case OP_EXPAND_DW:
        s = launch_expand_dw(src, batch, op.H, op.W, op.C, m.d_w + op.w_off, op.K, f32 + op.scale_off,
                             f32 + op.shift_off, op.act, m.d_w + op.w2_off, op.stride, f32 + op.scale2_off,
                             f32 + op.shift2_off, op.act2, (bf16*)dst, st);
        kind = KC_EXPAND_DW;
        fl = 2.0 * batch * op.H * op.W * (double)op.C * op.K + 2.0 * batch * op.Ho * op.Wo * op.K * 9;
        by = (double)batch * op.H * op.W * op.C * 2 + (double)op.K * op.C * 2 + 9.0 * op.K * 2 +
             (double)batch * op.Ho * op.Wo * op.K * 2;
        break;
      case OP_CONV_RGB:
        s = launch_conv2d_rgb(src, batch, op.H, op.W, m.d_w + op.w_off, op.K, op.R, op.stride, op.pad,
                              f32 + op.scale_off, f32 + op.shift_off, op.act, (bf16*)dst, st);
        kind = KC_DIRECT;
        fl = conv_flops(op, batch);
        by = conv_bytes(op, batch);
        break;
      case OP_CONV:
        s = launch_conv2d_ws(src, batch, op.H, op.W, op.C, m.d_w + op.w_off, op.K, op.R, op.S, op.stride, op.pad,
                             op.scale_off >= 0 ? f32 + op.scale_off : nullptr,
                             op.shift_off >= 0 ? f32 + op.shift_off : nullptr,
                             (const bf16*)bufp(op.res, d_in, d_out), op.act, dst, false, n_cu, ws.splitk,
                             ws.splitk_bytes, ws.tile_counters, st);
        kind = KC_MFMA;
        fl = conv_flops(op, batch);
        by = conv_bytes(op, batch);
        gm = batch * op.Ho * op.Wo;
        gn = op.K;
        gk = op.R * op.S * op.C;
        break;
      case OP_DW:
        s = launch_dwconv3x3(src, batch, op.H, op.W, op.C, m.d_w + op.w_off, op.stride, f32 + op.scale_off,
                             f32 + op.shift_off, op.act, (bf16*)dst, st);
        kind = KC_DW;
        fl = 2.0 * batch * op.Ho * op.Wo * op.C * 9;
        by = (double)batch * (op.H * op.W + op.Ho * op.Wo) * op.C * 2 + 9.0 * op.C * 2;
        break;
      case OP_MAXPOOL:
        s = launch_maxpool(src, batch, op.H, op.W, op.C, op.R, op.stride, op.pad, (bf16*)dst, st);
        by = (double)batch * (op.H * op.W + op.Ho * op.Wo) * op.C * 2;
        break;
      case OP_AVGPOOL:
        s = launch_avgpool(src, batch, op.H, op.W, op.C, (bf16*)dst, st);
        by = (double)batch * (op.H * op.W + 1) * op.C * 2;
        break;
      case OP_EMBED_LN:
        s = launch_embed_ln((const int*)src, batch * op.T, op.T, op.K, m.d_w + op.w_off, m.d_w + op.w2_off,
                            m.d_w + op.w3_off, op.C, nullptr, nullptr, 1e-12f, (bf16*)dst, st);
        by = (double)batch * op.T * (4 + 3.0 * op.C * 2 + op.C * 2);
        break;
      case OP_LAYERNORM:
        s = launch_layernorm(src, batch * op.H * op.W, op.C, nullptr, nullptr, 1e-12f, (bf16*)dst, st);
        by = (double)batch * op.H * op.W * op.C * 4;
        break;
      case OP_ATTENTION:
        s = launch_attention(src, batch, op.T, op.K, op.C / op.K, (bf16*)dst, st);
        kind = KC_ATTENTION;
        fl = 4.0 * batch * op.T * (double)op.T * op.C;
        by = (double)batch * op.T * op.C * 2 * 4;
        break;
      case OP_FC:
        s = launch_fc(src, batch, op.C, m.d_wp + op.wp_off, f32 + op.shift_off, op.K, op.act, dst, op.out_f32 != 0,
                      n_cu, ws.splitk, ws.splitk_bytes, st, true);
        kind = KC_FC;
        fl = 2.0 * batch * op.C * (double)op.K;
        by = (double)op.K * op.C * 2 + (double)batch * op.C * 2 + (double)batch * op.K * (op.out_f32 ? 4 : 2);
        break;
      default:
        break;
    }
    if (s != DSTACK_OK) return s;
    if (timer) timer->after(kind, fl, by, gm, gn, gk);
  }
  return DSTACK_OK;
}

void model_cost(const Model& m, int b, double* flops, double* mfma, double* wbytes, int* nk) {
  double f = 0, mf = 0;
  int n = 0;
  for (const Op& op : m.ops) {
    switch (op.kind) {
      case OP_CONV:
        f += conv_flops(op, b);
        mf += conv_flops(op, b);
        ++n;
        break;
      case OP_CONV_RGB:
        f += conv_flops(op, b);
        ++n;
        break;
      case OP_EXPAND_DW:
        f += 2.0 * b * op.H * op.W * (double)op.C * op.K + 2.0 * b * op.Ho * op.Wo * op.K * 9;
        mf += 2.0 * b * op.H * op.W * (double)op.C * op.K;
        ++n;
        break;
      case OP_DW:
        f += 2.0 * b * op.Ho * op.Wo * op.C * 9;
        ++n;
        break;
      case OP_FC:
        f += 2.0 * b * op.C * (double)op.K;
        ++n;
        break;
      case OP_ATTENTION:
        f += 4.0 * b * op.T * (double)op.T * op.C;
        ++n;
        break;
      case OP_LSTM: {
        double proj = 2.0 * op.T * b * op.I * 4.0 * op.Hd;
        double rec = 2.0 * op.T * b * op.Hd * 4.0 * op.Hd;
        f += proj + rec;
        mf += proj + rec;
        n += 1 + op.T;
        break;
      }
      default:
        ++n;
        break;
    }
  }
  double w = 0;
  for (const TensorSpec& t : m.tensors) w += 2.0 * t.numel;
  if (flops) *flops = f;
  if (mfma) *mfma = mf;
  if (wbytes) *wbytes = w;
  if (nk) *nk = n;
}

}  // namespace dstack
