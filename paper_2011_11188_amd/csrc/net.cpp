// mdnn_train_step: one minibatch SGD step of a fixed layer chain.
//
// Section 2.1 (tensors, a graph of ops, backpropagation) and section 3.1
// (minibatch SGD); storage types per section 3.2 (low-precision activations
// and working weights, fp32 accumulation and master weights).  The chain is
// fixed at creation; every op is enqueued on the caller's stream, nothing
// synchronises with the host, and all device memory is caller-owned.
//
// Workspace layout (each piece 256-byte aligned):
//   act[0]          low-precision copy of the input batch
//   act[i+1]        stored output of layer i (fp32 for the last layer)
//   argmax[i]       window index of each max-pool output
//   grad0, grad1    ping-pong buffers for activation gradients (low precision)
//   dz[i]           with fuse_update: the output gradient of each FC layer
//                   whose update runs in its weight-gradient product (it is
//                   read after the whole backward pass)
//   reduce_ws       split-K partials of the convolution backward-filter and
//                   of fp32 fully connected GEMMs, partial column sums of the
//                   bias gradients (the users run one after another)
#include <new>
#include <vector>

#include "internal.h"

using namespace mdnn;

struct LayerPlan {
  mdnn_layer_t L;
  int64_t w_off = 0, b_off = 0, nw = 0, nb = 0;
  int64_t in_feat = 0, out_feat = 0;  // per sample
  size_t out_off = 0;                 // act[i+1]
  size_t arg_off = 0;                 // pool argmax
  size_t cs_off = 0;                  // FC: bias-gradient partial column sums
  size_t cws_off = 0, cws_bytes = 0;  // conv: the filter gradient's own workspace
  bool input_relu = false;            // input produced by a ReLU (directly or through pooling)
  bool last = false;
  // fuse_update: this FC layer's weights are updated inside its weight-gradient
  // product (mdnn_gemm_tn_update); its output gradient lives at dz_off
  bool fuse_cand = false, fused = false;
  size_t dz_off = 0;
};

struct mdnn_net {
  std::vector<LayerPlan> layers;
  int64_t batch = 0;
  mdnn_train_cfg_t cfg{};
  mdnn_dtype_t lp = MDNN_F32;
  int64_t n_params = 0;
  int64_t in_feat = 0;
  size_t in_off = 0, g0_off = 0, g1_off = 0, fws_off = 0, fws_bytes = 0, ws_bytes = 0;
  // bound memory
  bool bound = false;
  float* master = nullptr;
  float* grads = nullptr;
  float* mom = nullptr;
  void* lowp = nullptr;
  char* ws = nullptr;
  mdnn_scaler_t* scaler = nullptr;
  // loss-scaled steps: the FC weight gradients are checked for non-finite
  // values by the GEMMs that write them and the FC bias gradients by the
  // pass that finishes their column sums; `unchecked` lists the other
  // gradient ranges (convolution layers) for a separate check.
  // prechecked is false when they do not fit in one CheckRanges (or the
  // batch is too tall for the batched column sums): then the update runs the
  // full check.
  bool prechecked = false;
  CheckRanges unchecked{};
  // fuse_update: whether any layer is fused (decided at bind time, from the
  // bound pointers) and the parameter ranges the SGD pass still updates
  bool fuse = false;
  CheckRanges rest{};
};

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static mdnn_conv_shape_t conv_shape(const mdnn_layer_t& L, int64_t batch) {
  return mdnn_conv_shape_t{batch, L.h, L.w, L.c_in, L.c_out, L.r, L.s, L.pad};
}

extern "C" mdnn_status_t mdnn_net_create(const mdnn_layer_t* layers, int32_t n_layers,
                                         int64_t batch, const mdnn_train_cfg_t* cfg,
                                         mdnn_net_t** out) {
  if (!layers || !cfg || !out) return fail(MDNN_ERR_NULL, "net_create: NULL argument");
  *out = nullptr;
  if (n_layers < 1 || n_layers > 256) return fail(MDNN_ERR_SHAPE, "net_create: 1..256 layers");
  if (batch < 1 || batch > (1 << 24)) return fail(MDNN_ERR_SHAPE, "net_create: bad batch");
  if (!dtype_ok(cfg->dtype)) return fail(MDNN_ERR_DTYPE, "net_create: unknown dtype");
  if (cfg->loss != MDNN_LOSS_XENT && cfg->loss != MDNN_LOSS_MSE)
    return fail(MDNN_ERR_SHAPE, "net_create: unknown loss");

  mdnn_net* net = new (std::nothrow) mdnn_net();
  if (!net) return fail(MDNN_ERR_SHAPE, "net_create: out of host memory");
  net->batch = batch;
  net->cfg = *cfg;
  net->lp = (mdnn_dtype_t)cfg->dtype;
  const size_t lps = dtype_size(net->lp);

  int64_t off = 0;
  bool prev_relu = false;
  // spatial output of the previous layer (h, w, c), or none
  bool prev_spatial = false;
  int64_t ph = 0, pw = 0, pc = 0, prev_out = -1;
  for (int i = 0; i < n_layers; ++i) {
    const mdnn_layer_t& L = layers[i];
    LayerPlan p;
    p.L = L;
    p.last = i == n_layers - 1;
    auto bad = [&](const char* why) {
      delete net;
      return fail(MDNN_ERR_SHAPE, "net_create: layer %d: %s", i, why);
    };
    if (L.act != MDNN_ACT_NONE && L.act != MDNN_ACT_RELU) return bad("unknown activation");
    if (L.kind == MDNN_LAYER_FC) {
      if (L.c_in < 1 || L.c_out < 1) return bad("FC sizes must be positive");
      p.in_feat = L.c_in;
      p.out_feat = L.c_out;
      p.nw = L.c_in * L.c_out;
      p.nb = L.c_out;
      prev_spatial = false;
    } else if (L.kind == MDNN_LAYER_CONV) {
      if (L.c_in < 1 || L.c_out < 1 || L.h < 1 || L.w < 1 || L.r < 1 || L.s < 1 || L.pad < 0)
        return bad("conv sizes must be positive");
      if (2 * L.pad != L.r - 1 || 2 * L.pad != L.s - 1) return bad("conv must keep the size (2*pad == r-1 == s-1)");
      if (prev_spatial && (ph != L.h || pw != L.w || pc != L.c_in)) return bad("conv input does not match");
      p.in_feat = L.h * L.w * L.c_in;
      p.out_feat = L.h * L.w * L.c_out;
      p.nw = L.c_out * L.r * L.s * L.c_in;
      p.nb = L.c_out;
      prev_spatial = true;
      ph = L.h; pw = L.w; pc = L.c_out;
    } else if (L.kind == MDNN_LAYER_MAXPOOL2) {
      if (L.c_in < 1 || L.h < 2 || L.w < 2 || (L.h & 1) || (L.w & 1)) return bad("maxpool needs even h, w >= 2");
      if (prev_spatial && (ph != L.h || pw != L.w || pc != L.c_in)) return bad("maxpool input does not match");
      if (p.last) return bad("the last layer must be FC or CONV");
      p.in_feat = L.h * L.w * L.c_in;
      p.out_feat = (L.h / 2) * (L.w / 2) * L.c_in;
      prev_spatial = true;
      ph = L.h / 2; pw = L.w / 2; pc = L.c_in;
    } else {
      return bad("unknown kind");
    }
    if (prev_out >= 0 && prev_out != p.in_feat) return bad("input size does not match the previous output");
    if (p.last && L.act != MDNN_ACT_NONE) return bad("the last layer has no activation");
    p.w_off = off;
    p.b_off = off + p.nw;
    off += p.nw + p.nb;
    p.input_relu = prev_relu;
    if (L.kind != MDNN_LAYER_MAXPOOL2) prev_relu = L.act == MDNN_ACT_RELU;
    prev_out = p.out_feat;
    net->layers.push_back(p);
  }
  net->n_params = off;
  net->in_feat = net->layers[0].in_feat;
  // (the batched bias column sums take at most 65535 row chunks)
  net->prechecked = true;
  for (const auto& p : net->layers)
    if (p.L.kind == MDNN_LAYER_FC && column_sums_chunks(batch, p.L.c_out, net->lp) > 65535) net->prechecked = false;
  for (const auto& p : net->layers) {
    int64_t o = 0, len = 0;
    if (p.L.kind == MDNN_LAYER_CONV) o = p.w_off, len = p.nw + p.nb;
    if (len == 0) continue;
    CheckRanges& r = net->unchecked;
    if (r.n > 0 && r.off[r.n - 1] + r.len[r.n - 1] == o) {
      r.len[r.n - 1] += len;  // adjacent to the previous range
    } else if (r.n < kMaxCheckRanges) {
      r.off[r.n] = o;
      r.len[r.n] = len;
      ++r.n;
    } else {
      net->prechecked = false;
    }
  }
  const LayerPlan& last = net->layers.back();
  if (cfg->loss == MDNN_LOSS_XENT && (last.out_feat != cfg->n_classes || cfg->n_classes > 1024)) {
    delete net;
    return fail(MDNN_ERR_SHAPE, "net_create: n_classes must equal the last layer's outputs (<= 1024)");
  }

  // workspace plan
  size_t w = 0;
  net->in_off = w;
  w = align256(w + (size_t)batch * net->in_feat * lps);
  int64_t max_feat = net->in_feat;
  size_t fws = 0;
  for (auto& p : net->layers) {
    p.out_off = w;
    w = align256(w + (size_t)batch * p.out_feat * (p.last ? 4 : lps));
    if (p.L.kind == MDNN_LAYER_MAXPOOL2) {
      p.arg_off = w;
      w = align256(w + (size_t)batch * p.out_feat);
    }
    if (p.L.kind == MDNN_LAYER_CONV) {
      // a region per layer: its partial sums stay until the backward pass
      // ends, when all layers' sums are finished in one launch
      mdnn_conv_shape_t cs = conv_shape(p.L, batch);
      p.cws_off = w;
      p.cws_bytes = mdnn_conv2d_bwd_filter_workspace(&cs, net->lp);
      w = align256(w + p.cws_bytes);
    }
    if (p.L.kind == MDNN_LAYER_FC) {
      const int64_t in = p.L.c_in, o = p.L.c_out;
      p.cs_off = w;
      w = align256(w + (size_t)column_sums_chunks(batch, o, net->lp) * o * 4);
      const size_t needs[4] = {mdnn_bias_act_bwd_workspace(batch, o), gemm_ws_bytes(net->lp, batch, o, in),
                               gemm_ws_bytes(net->lp, in, o, batch), gemm_ws_bytes(net->lp, batch, in, o)};
      for (size_t need : needs)
        if (need > fws) fws = need;
    }
    if (p.in_feat > max_feat) max_feat = p.in_feat;
    if (p.out_feat > max_feat) max_feat = p.out_feat;
  }
  // fuse_update candidates: FC layers whose weight gradient takes
  // mdnn_gemm_tn_update's shapes; fp16 storage when the loss is scaled
  // (finite fp16 operands give a finite fp32 product, so testing the
  // operands where they are stored -- the input batch's cast included --
  // tests the gradient)
  if (cfg->fuse_update && net->lp != MDNN_F32 && (!cfg->loss_scaling || net->lp == MDNN_F16)) {
    for (size_t i = 0; i < net->layers.size(); ++i) {
      LayerPlan& p = net->layers[i];
      if (p.L.kind != MDNN_LAYER_FC || p.L.c_in % 256 != 0 || p.L.c_out % 256 != 0 || batch % 64 != 0) continue;
      p.fuse_cand = true;
      p.dz_off = w;
      w = align256(w + (size_t)batch * p.L.c_out * lps);
    }
  }
  net->g0_off = w;
  w = align256(w + (size_t)batch * max_feat * lps);
  net->g1_off = w;
  w = align256(w + (size_t)batch * max_feat * lps);
  net->fws_off = w;
  net->fws_bytes = fws;
  w = align256(w + fws);
  net->ws_bytes = w;
  clear_error();
  *out = net;
  return MDNN_SUCCESS;
}

extern "C" mdnn_status_t mdnn_net_sizes(const mdnn_net_t* net, int64_t* n_params,
                                        size_t* workspace_bytes) {
  if (!net) return fail(MDNN_ERR_NULL, "net_sizes: NULL net");
  if (n_params) *n_params = net->n_params;
  if (workspace_bytes) *workspace_bytes = net->ws_bytes;
  return MDNN_SUCCESS;
}

extern "C" mdnn_status_t mdnn_net_bind(mdnn_net_t* net, float* master_w, float* grads,
                                       float* momentum, void* lowp_w, void* workspace,
                                       size_t workspace_bytes, mdnn_scaler_t* scaler) {
  if (!net) return fail(MDNN_ERR_NULL, "net_bind: NULL net");
  if (!master_w || !grads || !workspace) return fail(MDNN_ERR_NULL, "net_bind: master_w, grads and workspace are required");
  if (net->cfg.momentum != 0.0f && !momentum) return fail(MDNN_ERR_NULL, "net_bind: momentum buffer required");
  if (net->lp != MDNN_F32 && !lowp_w) return fail(MDNN_ERR_NULL, "net_bind: lowp_w required for a low-precision net");
  if (net->cfg.loss_scaling && !scaler) return fail(MDNN_ERR_NULL, "net_bind: scaler required with loss scaling");
  if (workspace_bytes < net->ws_bytes) return fail(MDNN_ERR_WORKSPACE, "net_bind: workspace needs %zu bytes", net->ws_bytes);
  if (!aligned(workspace, 256) || !aligned(master_w, 4) || !aligned(grads, 4) || (momentum && !aligned(momentum, 4)) ||
      (lowp_w && !aligned(lowp_w, dtype_size(net->lp))) || (scaler && !aligned(scaler, 4)))
    return fail(MDNN_ERR_MISALIGNED,
                "net_bind: workspace must be 256-byte aligned and parameter buffers aligned to their element size");
  net->master = master_w;
  net->grads = grads;
  net->mom = net->cfg.momentum != 0.0f ? momentum : nullptr;
  net->lowp = net->lp == MDNN_F32 ? nullptr : lowp_w;
  net->ws = (char*)workspace;
  net->scaler = net->cfg.loss_scaling ? scaler : nullptr;
  // fused layers: the candidates whose bound buffers fit the fused product
  // (a loss-scaled step needs the producer-side tests: prechecked)
  net->fuse = false;
  net->rest = CheckRanges{};
  const bool can_fuse = !net->scaler || net->prechecked;
  for (size_t i = 0; i < net->layers.size(); ++i) {
    LayerPlan& p = net->layers[i];
    p.fused = false;
    if (!p.fuse_cand || !can_fuse) continue;
    // dW[in, out] = X^T dZ with X = the stored input of layer i; only where
    // the unfused product would not split K (the fused one never does: the
    // same summation order keeps the step's results bit for bit)
    if (gemm_lp_splits(p.L.c_in, p.L.c_out, net->batch) > 1) continue;
    const char* x = net->ws + (i == 0 ? net->in_off : net->layers[i - 1].out_off);
    const char* wlp = (const char*)net->lowp + p.w_off * dtype_size(net->lp);
    p.fused = gemm_tn_update_ok(net->lp, p.L.c_in, p.L.c_out, net->batch, x, p.L.c_in, net->ws + p.dz_off,
                                p.L.c_out, net->master + p.w_off, net->mom ? net->mom + p.w_off : nullptr, wlp,
                                p.L.c_out);
    net->fuse |= p.fused;
  }
  if (net->fuse) {
    CheckRanges& r = net->rest;
    auto add = [&](int64_t o, int64_t len) {
      if (len == 0) return true;
      if (r.n > 0 && r.off[r.n - 1] + r.len[r.n - 1] == o) {
        r.len[r.n - 1] += len;
        return true;
      }
      if (r.n == kMaxCheckRanges) return false;
      r.off[r.n] = o;
      r.len[r.n] = len;
      ++r.n;
      return true;
    };
    bool ok = true;
    for (const auto& p : net->layers) {
      if (!p.fused) ok &= add(p.w_off, p.nw);
      ok &= add(p.b_off, p.nb);
    }
    if (!ok) {  // too fragmented: no fusion
      net->fuse = false;
      for (auto& p : net->layers) p.fused = false;
    }
  }
  net->bound = true;
  clear_error();
  return MDNN_SUCCESS;
}

extern "C" mdnn_status_t mdnn_net_sync_lowp(mdnn_net_t* net, mdnn_stream_t stream) {
  if (!net) return fail(MDNN_ERR_NULL, "net_sync_lowp: NULL net");
  if (!net->bound) return fail(MDNN_ERR_STATE, "net_sync_lowp: net not bound");
  if (!net->lowp) return MDNN_SUCCESS;
  return mdnn_cast(net->n_params, net->master, MDNN_F32, net->lowp, net->lp, stream);
}

extern "C" const void* mdnn_net_activation(const mdnn_net_t* net, int32_t i) {
  if (!net || !net->bound || i < 0 || i > (int32_t)net->layers.size()) return nullptr;
  if (i == 0) return net->ws + net->in_off;
  return net->ws + net->layers[i - 1].out_off;
}

extern "C" const void* mdnn_net_output_grad(const mdnn_net_t* net, int32_t which) {
  if (!net || !net->bound || (which != 0 && which != 1)) return nullptr;
  return net->ws + (which == 0 ? net->g0_off : net->g1_off);
}

extern "C" void mdnn_net_destroy(mdnn_net_t* net) { delete net; }

// One step; `async`: section 3.1's asynchronous variant, for nets that share
// their master weights with other nets stepping concurrently: the working
// copy is re-derived from the shared weights at the start of the step (an
// inconsistent snapshot while others update them), and the update is added
// to the shared weights with atomics instead of being written.
static mdnn_status_t run_step(mdnn_net_t* net, const float* x, const void* target, float* loss_out,
                              mdnn_stream_t stream, bool async) {
  if (!net) return fail(MDNN_ERR_NULL, "train_step: NULL net");
  if (!net->bound) return fail(MDNN_ERR_STATE, "train_step: net not bound");
  if (!x || !target || !loss_out) return fail(MDNN_ERR_NULL, "train_step: x, target and loss_out are required");
  if (!aligned(x, 4) || !aligned(target, 4) || !aligned(loss_out, 4))
    return fail(MDNN_ERR_MISALIGNED, "train_step: misaligned buffer");
  const int64_t B = net->batch;
  const mdnn_dtype_t lp = net->lp;
  char* ws = net->ws;
  const void* wlp = net->lowp ? net->lowp : (const void*)net->master;
  const size_t lps = dtype_size(lp);
  const float* scale = net->scaler ? &net->scaler->scale : nullptr;
  auto act_ptr = [&](size_t i) -> char* {
    return i == 0 ? ws + net->in_off : ws + net->layers[i - 1].out_off;
  };
  auto wptr = [&](const LayerPlan& p) { return (const char*)wlp + p.w_off * lps; };
  // FC weight gradients (and bias gradients) checked for the loss scaler as they are stored
  int32_t* nonfinite = (!async && net->scaler && net->prechecked) ? &net->scaler->reserved : nullptr;
  // fused updates (fuse_update): the activations and output gradients the
  // fused products read are tested where they are stored, and those
  // products run after every test of the step
  const bool fused = net->fuse && !async;
  int32_t* stored_flag = fused ? nonfinite : nullptr;

  // a1: input batch to the storage type (and, asynchronously, this worker's
  // snapshot of the shared weights)
  if (stored_flag && lp != MDNN_F32)
    MDNN_TRY(cast_f32_checked(B * net->in_feat, x, act_ptr(0), lp, stored_flag, as_stream(stream)));
  else
    MDNN_TRY(mdnn_cast(B * net->in_feat, x, MDNN_F32, act_ptr(0), lp, stream));
  if (async && net->lowp) MDNN_TRY(mdnn_cast(net->n_params, net->master, MDNN_F32, net->lowp, lp, stream));

  // forward
  for (size_t i = 0; i < net->layers.size(); ++i) {
    const LayerPlan& p = net->layers[i];
    const mdnn_dtype_t out_t = p.last ? MDNN_F32 : lp;
    const float* bias = net->master + p.b_off;
    const mdnn_act_t act = (mdnn_act_t)p.L.act;
    if (p.L.kind == MDNN_LAYER_FC) {
      MDNN_TRY(gemm_mixed_ws(MDNN_NN, B, p.L.c_out, p.L.c_in, 1.0f, act_ptr(i), p.L.c_in, wptr(p), p.L.c_out,
                             lp, 0.0f, nullptr, 0, act_ptr(i + 1), p.L.c_out, out_t, bias, act, nullptr, 0,
                             ws + net->fws_off, net->fws_bytes, stream, stored_flag));
    } else if (p.L.kind == MDNN_LAYER_CONV) {
      mdnn_conv_shape_t cs = conv_shape(p.L, B);
      MDNN_TRY(mdnn_conv2d_fwd(&cs, act_ptr(i), wptr(p), lp, bias, act, act_ptr(i + 1), out_t, stream));
    } else {
      MDNN_TRY(mdnn_maxpool2_fwd(B, p.L.h, p.L.w, p.L.c_in, act_ptr(i), act_ptr(i + 1),
                                 (uint8_t*)(ws + p.arg_off), lp, stream));
    }
  }

  // loss and its gradient (scaled by the loss scale), into grad0.  The
  // gradient with respect to the output of layer i goes to buffer
  // (L - 1 - i) % 2, or to its own buffer when layer i is fused.
  const size_t L = net->layers.size();
  auto dz_of = [&](size_t i) -> char* {
    if (fused && net->layers[i].fused) return ws + net->layers[i].dz_off;
    return ws + ((L - 1 - i) % 2 == 0 ? net->g0_off : net->g1_off);
  };
  char* gcur = dz_of(L - 1);
  const LayerPlan& last = net->layers.back();
  const float* out = (const float*)act_ptr(net->layers.size());
  // a classifier head's bias gradient comes out of the loss kernel itself
  const bool head_db = net->cfg.loss == MDNN_LOSS_XENT && last.L.kind == MDNN_LAYER_FC &&
                       softmax_xent_db_ok(B, last.out_feat) && (nonfinite || !net->scaler || async);
  if (net->cfg.loss == MDNN_LOSS_XENT) {
    if (head_db)
      MDNN_TRY(softmax_xent_db(B, last.out_feat, out, last.out_feat, (const int32_t*)target, scale, loss_out, gcur,
                               last.out_feat, lp, net->grads + last.b_off, nonfinite, as_stream(stream)));
    else
      MDNN_TRY(mdnn_softmax_xent(B, last.out_feat, out, last.out_feat, (const int32_t*)target, scale,
                                 loss_out, gcur, last.out_feat, lp, stream));
  } else {
    MDNN_TRY(mdnn_mse_loss(B, last.out_feat, out, (const float*)target, scale, loss_out, gcur, lp,
                           stream));
  }

  // backward
  // loss-scaled FC bias gradients: partial column sums per layer now, all
  // layers finished (and checked) in one launch after the loop
  ColsumBatch bias_sums{};
  // fused layers' output gradients stay in their own buffers: their partial
  // sums go in one batched launch after the loop
  StripBatch strips{};
  // convolution layers' weight and bias sums: second passes in one launch
  // after the loop
  ReduceBatch conv_sums{};
  for (size_t ii = net->layers.size(); ii-- > 0;) {
    const LayerPlan& p = net->layers[ii];
    const char* a_in = act_ptr(ii);
    gcur = dz_of(ii);
    char* gnxt = ii > 0 ? dz_of(ii - 1) : nullptr;
    float* gw = net->grads + p.w_off;
    float* gb = net->grads + p.b_off;
    const void* mask = p.input_relu ? (const void*)a_in : nullptr;
    if (p.L.kind == MDNN_LAYER_FC) {
      const int64_t in = p.L.c_in, o = p.L.c_out;
      // bias gradient first, while dZ (just written) is still in the caches
      if (head_db && ii + 1 == net->layers.size()) {
        // done by the loss kernel
      } else if (nonfinite) {
        float* part = (float*)(ws + p.cs_off);
        if (fused && p.fused && strips.n < kMaxColsumBatch && column_sums_strip_ok(gcur, lp, o, part)) {
          strips.x[strips.n] = (const uint16_t*)gcur;
          strips.partial[strips.n] = part;
          strips.cols[strips.n] = o;
          ++strips.n;
        } else {
          MDNN_TRY(column_sums_partial(gcur, lp, B, o, part, as_stream(stream)));
        }
        if (bias_sums.n == kMaxColsumBatch) {
          MDNN_TRY(column_sums_partial_batch(strips, lp, B, as_stream(stream)));
          strips.n = 0;
          MDNN_TRY(column_sums_final(bias_sums, nonfinite, as_stream(stream)));
          bias_sums.n = 0;
        }
        const int e = bias_sums.n++;
        bias_sums.part[e] = part;
        bias_sums.out[e] = gb;
        bias_sums.chunks[e] = column_sums_chunks(B, o, lp);
        bias_sums.cols[e] = o;
      } else {
        MDNN_TRY(mdnn_bias_act_bwd(B, o, gcur, nullptr, MDNN_ACT_NONE, nullptr, gb, lp, ws + net->fws_off,
                                   net->fws_bytes, stream));
      }
      // dW[in, out] = X^T dZ  (TN: A = X stored [B, in], B = dZ stored [B, out]); a fused
      // layer's product runs after the backward pass, updating the weights
      if (!(fused && p.fused))
        MDNN_TRY(gemm_mixed_ws(MDNN_TN, in, o, B, 1.0f, a_in, in, gcur, o, lp, 0.0f, nullptr, 0, gw, o, MDNN_F32,
                               nullptr, MDNN_ACT_NONE, nullptr, 0, ws + net->fws_off, net->fws_bytes, stream,
                               nonfinite));
      if (ii > 0) {
        // dX[B, in] = dZ W^T, masked by the input's ReLU  (NT: B operand = W stored [in, out])
        MDNN_TRY(gemm_mixed_ws(MDNN_NT, B, in, o, 1.0f, gcur, o, wptr(p), o, lp, 0.0f, nullptr, 0, gnxt, in, lp,
                               nullptr, MDNN_ACT_NONE, mask, in, ws + net->fws_off, net->fws_bytes, stream,
                               stored_flag));
      }
    } else if (p.L.kind == MDNN_LAYER_CONV) {
      mdnn_conv_shape_t cs = conv_shape(p.L, B);
      MDNN_TRY(conv2d_bwd_filter_deferred(&cs, a_in, gcur, lp, gw, gb, ws + p.cws_off, p.cws_bytes,
                                          as_stream(stream), &conv_sums));
      if (ii > 0)
        MDNN_TRY(mdnn_conv2d_bwd_data(&cs, gcur, wptr(p), lp, mask, gnxt, lp, stream));
    } else {
      MDNN_TRY(mdnn_maxpool2_bwd(B, p.L.h, p.L.w, p.L.c_in, gcur, (const uint8_t*)(ws + p.arg_off),
                                 gnxt, lp, stream));
    }
  }

  MDNN_TRY(reduce_batch_launch(conv_sums, as_stream(stream)));
  MDNN_TRY(column_sums_partial_batch(strips, lp, B, as_stream(stream)));
  MDNN_TRY(column_sums_final(bias_sums, nonfinite, as_stream(stream)));
  if (fused) {
    // every test of this step is done: the fused layers' weight gradients,
    // each applied to its weights as it is produced, then the update of the
    // other parameters (and the scaler's state)
    if (nonfinite) MDNN_TRY(finite_check_ranges(net->grads, net->unchecked, net->scaler, as_stream(stream)));
    for (size_t ii = 0; ii < L; ++ii) {
      const LayerPlan& p = net->layers[ii];
      if (!p.fused) continue;
      MDNN_TRY(mdnn_gemm_tn_update(p.L.c_in, p.L.c_out, B, act_ptr(ii), p.L.c_in, dz_of(ii), p.L.c_out, lp,
                                   net->master + p.w_off, net->mom ? net->mom + p.w_off : nullptr,
                                   (char*)net->lowp + p.w_off * lps, p.L.c_out, net->cfg.lr, net->cfg.momentum,
                                   net->scaler, stream));
    }
    return sgd_update_ranges_prechecked(net->rest, net->master, net->grads, net->mom, net->lowp, lp, net->cfg.lr,
                                        net->cfg.momentum, net->scaler, as_stream(stream));
  }

  // update (and the low-precision working copy)
  if (async)
    return mdnn_sgd_update_async(net->n_params, net->master, net->grads, net->mom, net->cfg.lr,
                                 net->cfg.momentum, net->scaler, stream);
  if (nonfinite) {
    MDNN_TRY(finite_check_ranges(net->grads, net->unchecked, net->scaler, as_stream(stream)));
    return sgd_update_prechecked(net->n_params, net->master, net->grads, net->mom, net->lowp, lp, net->cfg.lr,
                                 net->cfg.momentum, net->scaler, stream);
  }
  return mdnn_sgd_update(net->n_params, net->master, net->grads, net->mom, net->lowp, lp,
                         net->cfg.lr, net->cfg.momentum, net->scaler, stream);
}

extern "C" mdnn_status_t mdnn_train_step(mdnn_net_t* net, const float* x, const void* target,
                                         float* loss_out, mdnn_stream_t stream) {
  return run_step(net, x, target, loss_out, stream, false);
}

extern "C" mdnn_status_t mdnn_train_step_async(mdnn_net_t* net, const float* x, const void* target,
                                               float* loss_out, mdnn_stream_t stream) {
  return run_step(net, x, target, loss_out, stream, true);
}

// ---------------------------------------------------------------------------
// Recorded steps: one mdnn_train_step captured into a HIP graph, replayed
// with a single launch (the small configurations are bound by launch
// latency, not by their kernels).
// ---------------------------------------------------------------------------
struct mdnn_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

extern "C" mdnn_status_t mdnn_train_graph_create(mdnn_net_t* net, const float* x, const void* target,
                                                 float* loss_out, mdnn_graph_t** out) {
  if (!out) return fail(MDNN_ERR_NULL, "train_graph_create: out is NULL");
  *out = nullptr;
  if (!net) return fail(MDNN_ERR_NULL, "train_graph_create: NULL net");
  if (!net->bound) return fail(MDNN_ERR_STATE, "train_graph_create: net not bound");
  // capture on a private stream (the legacy default stream cannot be captured)
  hipStream_t s = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  if (e != hipSuccess) return fail(MDNN_ERR_LAUNCH, "train_graph_create: stream: %s", hipGetErrorString(e));
  e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    (void)hipStreamDestroy(s);
    return fail(MDNN_ERR_LAUNCH, "train_graph_create: begin capture: %s", hipGetErrorString(e));
  }
  const mdnn_status_t st = run_step(net, x, target, loss_out, (mdnn_stream_t)s, false);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(s, &graph);  // always end the capture, also after a failed step
  (void)hipStreamDestroy(s);
  if (st != MDNN_SUCCESS) {
    if (graph) (void)hipGraphDestroy(graph);
    return st;  // the step's own message stays
  }
  if (e != hipSuccess || !graph)
    return fail(MDNN_ERR_LAUNCH, "train_graph_create: end capture: %s", hipGetErrorString(e));
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    (void)hipGraphDestroy(graph);
    return fail(MDNN_ERR_LAUNCH, "train_graph_create: instantiate: %s", hipGetErrorString(e));
  }
  mdnn_graph_t* g = new (std::nothrow) mdnn_graph_t;
  if (!g) {
    (void)hipGraphExecDestroy(exec);
    (void)hipGraphDestroy(graph);
    return fail(MDNN_ERR_STATE, "train_graph_create: out of host memory");
  }
  g->graph = graph;
  g->exec = exec;
  *out = g;
  clear_error();
  return MDNN_SUCCESS;
}

extern "C" mdnn_status_t mdnn_graph_launch(mdnn_graph_t* g, mdnn_stream_t stream) {
  if (!g || !g->exec) return fail(MDNN_ERR_NULL, "graph_launch: NULL graph");
  const hipError_t e = hipGraphLaunch(g->exec, as_stream(stream));
  if (e != hipSuccess) return fail(MDNN_ERR_LAUNCH, "graph_launch: %s", hipGetErrorString(e));
  return MDNN_SUCCESS;
}

extern "C" void mdnn_graph_destroy(mdnn_graph_t* g) {
  if (!g) return;
  if (g->exec) (void)hipGraphExecDestroy(g->exec);
  if (g->graph) (void)hipGraphDestroy(g->graph);
  delete g;
}
