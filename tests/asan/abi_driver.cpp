// Drives libsagips's C ABI on the CPU, against the stub HIP runtime, under the
// address and undefined-behaviour sanitizers: every documented error path of
// every entry point (each must return its status and a message, never abort),
// and valid calls of every entry point (argument checks, workspace sizing and
// the host side of every launcher, whose launch shapes the stub checks).
// Device pointers are addresses of an unmapped region: the library's host
// code must never dereference them.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <functional>
#include <string>
#include <vector>

#include "sagips.h"

extern "C" {
void stub_set_arch(const char* arch);
long stub_launches();
long stub_bad_launches();
long stub_live_events();
long stub_live_allocs();
}

namespace {

int g_fail = 0, g_checks = 0;

// Fake device memory: 16-byte aligned addresses far from anything mapped, 1 MiB
// apart (buffers larger than that get their own distant offsets).
template <class T = float>
T* dev(uint64_t off) {
  return reinterpret_cast<T*>((uintptr_t)0x7e0000000000ull + (off << 20));
}

void expect(const char* what, sagips_status got, sagips_status want, sagips_ctx* c) {
  ++g_checks;
  const char* msg = sagips_last_error(c);
  if (got != want || !msg) {
    ++g_fail;
    printf("FAIL %s: status %d, expected %d (%s)\n", what, (int)got, (int)want, msg ? msg : "(null message)");
  } else if (want != SAGIPS_OK && strlen(msg) == 0) {
    ++g_fail;
    printf("FAIL %s: empty message\n", what);
  }
}

sagips_source source(int n_theta, int d, int64_t E) {
  sagips_source s;
  memset(&s, 0, sizeof(s));
  s.theta = dev(1);
  s.n_theta = n_theta;
  s.d = d;
  s.events_per_theta = E;
  s.seed = 7;
  return s;
}

sagips_mlp mlp(std::vector<int> widths, int prec, int feat) {
  sagips_mlp m;
  memset(&m, 0, sizeof(m));
  m.n_layers = (int)widths.size() - 1;
  for (size_t i = 0; i < widths.size(); ++i) m.width[i] = widths[i];
  for (int l = 0; l < m.n_layers; ++l) {
    m.W[l] = dev(100 + 2 * l);
    m.b[l] = dev(101 + 2 * l);
  }
  m.leaky_slope = 0.2f;
  m.precision = prec;
  m.features = feat;
  return m;
}

sagips_disc_out outs(int n_layers, bool grads, bool theta) {
  sagips_disc_out o;
  memset(&o, 0, sizeof(o));
  o.logits_fake = dev(200);
  o.logits_real = dev(201);
  o.loss_d = dev(202);
  o.loss_g = dev(203);
  o.dLg_dx = dev(204);
  if (theta) o.dLg_dtheta = dev(205);
  for (int l = 0; grads && l < n_layers; ++l) {
    o.dW[l] = dev(210 + 2 * l);
    o.db[l] = dev(211 + 2 * l);
  }
  return o;
}

sagips_gen gen(int M, std::vector<int> widths) {
  sagips_gen g;
  memset(&g, 0, sizeof(g));
  g.n_layers = (int)widths.size() - 1;
  for (size_t i = 0; i < widths.size(); ++i) g.width[i] = widths[i];
  for (int l = 0; l < g.n_layers; ++l) {
    g.W[l] = dev(300 + 2 * l);
    g.b[l] = dev(301 + 2 * l);
  }
  g.n_members = M;
  g.leaky_slope = 0.2f;
  return g;
}

}  // namespace

int main() {
  const sagips_status OK = SAGIPS_OK, INVAL = SAGIPS_E_INVAL, UNSUP = SAGIPS_E_UNSUPPORTED;
  if (!sagips_last_error(nullptr)) { printf("FAIL last_error(NULL) is NULL\n"); return 1; }

  // ---- context creation
  sagips_ctx* c = nullptr;
  expect("create(out=NULL)", sagips_create(nullptr, 0, nullptr), INVAL, nullptr);
  expect("create(device=-1)", sagips_create(&c, -1, nullptr), INVAL, nullptr);
  expect("create(device=1 of 1)", sagips_create(&c, 1, nullptr), INVAL, nullptr);
  stub_set_arch("gfx942");
  expect("create on gfx942", sagips_create(&c, 0, nullptr), SAGIPS_E_ARCH, nullptr);
  if (c) { printf("FAIL create left a context on failure\n"); ++g_fail; }
  stub_set_arch("gfx950");

  // ---- every call with a NULL context
  sagips_source s0 = source(4, 2, 1000);
  sagips_mlp m0 = mlp({2, 128, 128, 128, 1}, SAGIPS_F32, SAGIPS_FEAT_IDENTITY);
  sagips_disc_out o0 = outs(4, true, true);
  sagips_gen g0 = gen(1, {6, 128, 128, 128, 128, 6});
  sagips_param_set ps0;
  memset(&ps0, 0, sizeof(ps0));
  expect("sample(NULL ctx)", sagips_sample_events(nullptr, &s0, dev(1000), nullptr), INVAL, nullptr);
  expect("disc(NULL ctx)", sagips_disc_fwd_bwd(nullptr, &m0, nullptr, &s0, 4000, dev(1001), 4000, &o0), INVAL, nullptr);
  expect("disc_noalloc(NULL ctx)", sagips_disc_fwd_bwd_noalloc(nullptr, &m0, nullptr, &s0, 4000, dev(1001), 4000, &o0),
         INVAL, nullptr);
  expect("param_grad(NULL ctx)", sagips_param_grad(nullptr, &s0, SAGIPS_CRITIC_QUADRATIC, nullptr, dev(1002), nullptr),
         INVAL, nullptr);
  expect("bootstrap(NULL ctx)", sagips_bootstrap(nullptr, dev(1003), 100, 2, 1, 0, 50, dev(1004), nullptr), INVAL, nullptr);
  expect("bootstrap_rows(NULL ctx)", sagips_bootstrap_rows(nullptr, dev(1003), 100, 2, 1, 0, 50, dev(1004), nullptr),
         INVAL, nullptr);
  expect("gen_forward(NULL ctx)", sagips_gen_forward(nullptr, &g0, dev(1005), 16, dev(1006)), INVAL, nullptr);
  expect("ensemble(NULL ctx)", sagips_ensemble_response(nullptr, &g0, dev(1005), 16, nullptr, dev(1007), dev(1008), nullptr),
         INVAL, nullptr);
  expect("adam(NULL ctx)", sagips_adam_step(nullptr, &ps0, 1, 1e-3, 0.9, 0.999, 1e-8), INVAL, nullptr);
  expect("set_stream(NULL ctx)", sagips_set_stream(nullptr, nullptr), INVAL, nullptr);
  expect("set_timing(NULL ctx)", sagips_set_timing(nullptr, 1), INVAL, nullptr);
  expect("set_bf16_chunk_rows(NULL ctx)", sagips_set_bf16_chunk_rows(nullptr, 128), INVAL, nullptr);
  expect("destroy(NULL)", sagips_destroy(nullptr), OK, nullptr);

  expect("create", sagips_create(&c, 0, nullptr), OK, nullptr);
  if (!c) { printf("FAIL no context\n"); return 1; }

  // ---- sample_events
  {
    sagips_source s = source(4, 2, 1000);
    expect("sample ok", sagips_sample_events(c, &s, dev(1000), nullptr), OK, c);
    expect("sample words only", sagips_sample_events(c, &s, nullptr, dev<uint32_t>(1010)), OK, c);
    expect("sample no outputs", sagips_sample_events(c, &s, nullptr, nullptr), INVAL, c);
    expect("sample src NULL", sagips_sample_events(c, nullptr, dev(1000), nullptr), INVAL, c);
    expect("sample x misaligned", sagips_sample_events(c, &s, dev(1000) + 1, nullptr), INVAL, c);
    sagips_source t = s; t.theta = nullptr;
    expect("sample theta NULL", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.theta = reinterpret_cast<const float*>(reinterpret_cast<uintptr_t>(dev(1)) + 2);
    expect("sample theta 2-byte aligned", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.theta = dev(1) + 1;
    expect("sample theta 4-byte aligned (a shard's rows)", sagips_sample_events(c, &t, dev(1000), nullptr), OK, c);
    t = s; t.n_theta = 0;
    expect("sample n_theta 0", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.n_theta = 65536;
    expect("sample n_theta 65536", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.d = 4;
    expect("sample d 4", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.events_per_theta = 0;
    expect("sample E 0", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.n_theta = 1024; t.events_per_theta = (int64_t)1 << 21;
    expect("sample N = 2^31", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = s; t.counter_base = UINT64_MAX - 100;
    expect("sample counter overflow", sagips_sample_events(c, &t, dev(1000), nullptr), INVAL, c);
    t = source(64, 2, (int64_t)1 << 22);
    expect("sample stress size", sagips_sample_events(c, &t, dev(1000), nullptr), OK, c);
  }

  // ---- param_grad
  {
    sagips_source s = source(64, 2, (int64_t)1 << 22);
    expect("param_grad quadratic", sagips_param_grad(c, &s, SAGIPS_CRITIC_QUADRATIC, nullptr, dev(1100), dev(1101)), OK, c);
    expect("param_grad buffer", sagips_param_grad(c, &s, SAGIPS_CRITIC_BUFFER, dev(1102), dev(1100), nullptr), OK, c);
    expect("param_grad no output", sagips_param_grad(c, &s, SAGIPS_CRITIC_QUADRATIC, nullptr, nullptr, nullptr), INVAL, c);
    expect("param_grad buffer without dL_dx", sagips_param_grad(c, &s, SAGIPS_CRITIC_BUFFER, nullptr, dev(1100), nullptr),
           INVAL, c);
    expect("param_grad buffer with loss", sagips_param_grad(c, &s, SAGIPS_CRITIC_BUFFER, dev(1102), dev(1100), dev(1101)),
           INVAL, c);
    expect("param_grad quadratic with dL_dx",
           sagips_param_grad(c, &s, SAGIPS_CRITIC_QUADRATIC, dev(1102), dev(1100), nullptr), INVAL, c);
    expect("param_grad critic 7", sagips_param_grad(c, &s, (sagips_critic)7, nullptr, dev(1100), nullptr), INVAL, c);
    expect("param_grad dL_dx misaligned",
           sagips_param_grad(c, &s, SAGIPS_CRITIC_BUFFER, dev(1102) + 2, dev(1100), nullptr), INVAL, c);
  }

  // ---- discriminator step, fp32
  {
    sagips_source s = source(32, 2, 8192);
    sagips_mlp m = mlp({2, 128, 128, 128, 1}, SAGIPS_F32, SAGIPS_FEAT_IDENTITY);
    sagips_disc_out o = outs(4, true, true);
    expect("disc small", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200), 262144, &o), OK, c);
    expect("disc small no-alloc", sagips_disc_fwd_bwd_noalloc(c, &m, nullptr, &s, 262144, dev(1200), 262144, &o), OK, c);
    sagips_source e = source(40, 2, 50);   // E < tile: sampled into the workspace first
    expect("disc split path", sagips_disc_fwd_bwd(c, &m, nullptr, &e, 2000, dev(1200), 1000, &o), OK, c);
    sagips_disc_out og = outs(4, false, false);
    expect("disc buffer fake", sagips_disc_fwd_bwd(c, &m, dev(1201), nullptr, 5000, dev(1200), 3000, &og), OK, c);
    expect("disc D NULL", sagips_disc_fwd_bwd(c, nullptr, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    expect("disc out NULL", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200), 262144, nullptr), INVAL, c);
    expect("disc both fakes", sagips_disc_fwd_bwd(c, &m, dev(1201), &s, 262144, dev(1200), 262144, &o), INVAL, c);
    expect("disc no fake", sagips_disc_fwd_bwd(c, &m, nullptr, nullptr, 262144, dev(1200), 262144, &o), INVAL, c);
    expect("disc real NULL", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, nullptr, 262144, &o), INVAL, c);
    expect("disc real misaligned", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200) + 1, 262144, &o), INVAL, c);
    expect("disc n_real 0", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200), 0, &o), INVAL, c);
    expect("disc n_real 2^30", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200), (int64_t)1 << 30, &o), INVAL, c);
    expect("disc n_fake mismatch", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 1000, dev(1200), 1000, &o), INVAL, c);
    expect("disc dtheta without source", sagips_disc_fwd_bwd(c, &m, dev(1201), nullptr, 1000, dev(1200), 1000, &o), INVAL, c);
    sagips_disc_out op = o; op.db[2] = nullptr;
    expect("disc dW/db partly given", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 262144, dev(1200), 262144, &op), INVAL, c);
    sagips_mlp t = m; t.n_layers = 1;
    expect("disc one layer", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.W[1] = nullptr;
    expect("disc W NULL", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.b[2] = dev(1300) + 1;
    expect("disc b misaligned", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.width[4] = 2;
    expect("disc last width 2", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.width[2] = 0;
    expect("disc width 0", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.features = 9;
    expect("disc features 9", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.precision = 5;
    expect("disc precision 5", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.features = SAGIPS_FEAT_HD8;
    expect("disc HD8 with d 2", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    t = m; t.width[0] = 3;
    expect("disc width[0] != d", sagips_disc_fwd_bwd(c, &t, nullptr, &s, 262144, dev(1200), 262144, &o), INVAL, c);
    sagips_mlp w96 = mlp({2, 96, 96, 1}, SAGIPS_F32, SAGIPS_FEAT_IDENTITY);
    sagips_disc_out o96 = outs(3, true, true);
    expect("disc fp32 width 96", sagips_disc_fwd_bwd(c, &w96, nullptr, &s, 262144, dev(1200), 262144, &o96), UNSUP, c);
    sagips_mlp deep = mlp({2, 128, 128, 128, 128, 128, 1}, SAGIPS_F32, SAGIPS_FEAT_IDENTITY);
    sagips_disc_out od = outs(6, true, true);
    expect("disc fp32 too deep", sagips_disc_fwd_bwd(c, &deep, nullptr, &s, 262144, dev(1200), 262144, &od), UNSUP, c);
    // the paper's network on its two observables
    sagips_source p = source(1024, 3, 100);
    sagips_mlp pm = mlp({2, 128, 128, 128, 128, 1}, SAGIPS_F32, SAGIPS_FEAT_PROXY2);
    sagips_disc_out po = outs(5, true, true);
    expect("disc paper shape", sagips_disc_fwd_bwd(c, &pm, nullptr, &p, 102400, dev(1200), 102400, &po), OK, c);
    expect("disc paper shape no-alloc", sagips_disc_fwd_bwd_noalloc(c, &pm, nullptr, &p, 102400, dev(1200), 102400, &po),
           OK, c);
    sagips_source big = source(8192, 2, 8192);
    expect("disc no-alloc beyond the scratch",
           sagips_disc_fwd_bwd_noalloc(c, &m, nullptr, &big, (int64_t)1 << 26, dev(1200), 65536, &o), INVAL, c);
  }

  // ---- discriminator step, bf16
  {
    sagips_source s = source(3, 2, 1000);
    sagips_mlp m = mlp({2, 256, 256, 256, 256, 1}, SAGIPS_BF16, SAGIPS_FEAT_IDENTITY);
    sagips_disc_out o = outs(5, true, true);
    expect("bf16 medium reduced", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 3000, dev(1400), 2999, &o), OK, c);
    expect("bf16 chunk rows 127", sagips_set_bf16_chunk_rows(c, 127), INVAL, c);
    expect("bf16 chunk rows 200", sagips_set_bf16_chunk_rows(c, 200), INVAL, c);
    expect("bf16 chunk rows too many", sagips_set_bf16_chunk_rows(c, ((int64_t)1 << 22) + 128), INVAL, c);
    expect("bf16 chunk rows 1024", sagips_set_bf16_chunk_rows(c, 1024), OK, c);
    expect("bf16 medium in chunks", sagips_disc_fwd_bwd(c, &m, nullptr, &s, 3000, dev(1400), 2999, &o), OK, c);
    expect("bf16 chunk rows default", sagips_set_bf16_chunk_rows(c, 0), OK, c);
    sagips_source h = source(2, 3, 777);
    sagips_mlp hm = mlp({8, 512, 512, 512, 512, 1}, SAGIPS_BF16, SAGIPS_FEAT_HD8);
    expect("bf16 higher-dim reduced", sagips_disc_fwd_bwd(c, &hm, nullptr, &h, 1554, dev(1400), 1500, &o), OK, c);
    sagips_source full = source(256, 2, 16384);
    expect("bf16 medium full size: workspace beyond the device",
           sagips_disc_fwd_bwd(c, &m, nullptr, &full, 4194304, dev(1400), 4194304, &o), SAGIPS_E_NOMEM, c);
    expect("bf16 no-alloc beyond the scratch", sagips_disc_fwd_bwd_noalloc(c, &m, nullptr, &s, 3000, dev(1400), 2999, &o),
           INVAL, c);
    sagips_mlp w128 = mlp({2, 128, 128, 1}, SAGIPS_BF16, SAGIPS_FEAT_IDENTITY);
    sagips_disc_out o3 = outs(3, true, true);
    expect("bf16 width 128", sagips_disc_fwd_bwd(c, &w128, nullptr, &s, 3000, dev(1400), 2999, &o3), UNSUP, c);
    sagips_mlp px = mlp({2, 256, 256, 1}, SAGIPS_BF16, SAGIPS_FEAT_PROXY2);
    sagips_source p3 = source(3, 3, 1000);
    expect("bf16 proxy2", sagips_disc_fwd_bwd(c, &px, nullptr, &p3, 3000, dev(1400), 2999, &o3), UNSUP, c);
    sagips_mlp slope = m; slope.leaky_slope = 1.5f;
    expect("bf16 slope 1.5", sagips_disc_fwd_bwd(c, &slope, nullptr, &s, 3000, dev(1400), 2999, &o), UNSUP, c);
  }

  // ---- bootstrap draws
  {
    // the pool (up to 1 GiB) at unit 1500, outputs from unit 4000 on
    expect("bootstrap ok", sagips_bootstrap(c, dev(1500), 8388608, 2, 5, 3, 4194304, dev(4000), dev<int64_t>(5000)), OK, c);
    expect("bootstrap rows ok", sagips_bootstrap_rows(c, dev(1500), 8388608, 2, 5, 3, 4194304, dev(4000), nullptr), OK, c);
    expect("bootstrap data NULL", sagips_bootstrap(c, nullptr, 100, 2, 5, 3, 50, dev(1600), nullptr), INVAL, c);
    expect("bootstrap d 4", sagips_bootstrap(c, dev(1500), 100, 4, 5, 3, 50, dev(1600), nullptr), INVAL, c);
    expect("bootstrap n_data 0", sagips_bootstrap(c, dev(1500), 0, 2, 5, 3, 50, dev(1600), nullptr), INVAL, c);
    expect("bootstrap n_data 2^32 + 1",
           sagips_bootstrap(c, dev(1500), ((int64_t)1 << 32) + 1, 2, 5, 3, 50, dev(100000), nullptr), INVAL, c);
    expect("bootstrap n_out 0", sagips_bootstrap(c, dev(1500), 100, 2, 5, 3, 0, dev(1600), nullptr), INVAL, c);
    expect("bootstrap out misaligned", sagips_bootstrap(c, dev(1500), 100, 2, 5, 3, 50, dev(1600) + 1, nullptr), INVAL, c);
    expect("bootstrap out overlaps data", sagips_bootstrap(c, dev(1500), 100, 2, 5, 3, 50, dev(1500) + 100, nullptr), INVAL, c);
    expect("bootstrap idx overlaps out",
           sagips_bootstrap(c, dev(1500), 100, 2, 5, 3, 50, dev(1600), reinterpret_cast<int64_t*>(dev(1600))), INVAL, c);
    expect("bootstrap rows pool beyond 2^27",
           sagips_bootstrap_rows(c, dev(1500), ((int64_t)1 << 27) + 1, 2, 5, 3, 50, dev(4000), nullptr), UNSUP, c);
  }

  // ---- generator, ensemble, optimiser
  {
    sagips_gen g = gen(100, {6, 128, 128, 128, 128, 6});
    expect("gen_forward ok", sagips_gen_forward(c, &g, dev(1800), 1024, dev(1801)), OK, c);
    float* dW[SAGIPS_MAX_LAYERS] = {};
    float* db[SAGIPS_MAX_LAYERS] = {};
    for (int l = 0; l < g.n_layers; ++l) { dW[l] = dev(1810 + 2 * l); db[l] = dev(1811 + 2 * l); }
    expect("gen_backward ok", sagips_gen_backward(c, &g, dev(1800), 1024, dev(1802), dW, db), OK, c);
    expect("ensemble ok", sagips_ensemble_response(c, &g, dev(1800), 1024, dev(1803), dev(1804), dev(1805), dev(1806)), OK, c);
    expect("gen G NULL", sagips_gen_forward(c, nullptr, dev(1800), 1024, dev(1801)), INVAL, c);
    expect("gen noise NULL", sagips_gen_forward(c, &g, nullptr, 1024, dev(1801)), INVAL, c);
    expect("gen theta NULL", sagips_gen_forward(c, &g, dev(1800), 1024, nullptr), INVAL, c);
    expect("gen k 0", sagips_gen_forward(c, &g, dev(1800), 0, dev(1801)), INVAL, c);
    sagips_gen t = g; t.n_members = 0;
    expect("gen no members", sagips_gen_forward(c, &t, dev(1800), 1024, dev(1801)), INVAL, c);
    t = g; t.n_layers = 1;
    expect("gen one layer", sagips_gen_forward(c, &t, dev(1800), 1024, dev(1801)), INVAL, c);
    t = g; t.W[2] = dev(1900) + 3;
    expect("gen W misaligned", sagips_gen_forward(c, &t, dev(1800), 1024, dev(1801)), INVAL, c);
    sagips_gen w64 = gen(1, {6, 64, 64, 6});
    expect("gen hidden 64", sagips_gen_forward(c, &w64, dev(1800), 1024, dev(1801)), UNSUP, c);
    dW[1] = nullptr;
    expect("gen_backward dW NULL", sagips_gen_backward(c, &g, dev(1800), 1024, dev(1802), dW, db), INVAL, c);
    expect("ensemble p_true without r_hat",
           sagips_ensemble_response(c, &g, dev(1800), 1024, dev(1803), dev(1804), dev(1805), nullptr), INVAL, c);
    sagips_gen huge = gen(65535, {6, 128, 128, 128, 128, 6});
    expect("ensemble M k out >= 2^31",
           sagips_ensemble_response(c, &huge, dev(1800), 8192, nullptr, dev(1804), dev(1805), nullptr), INVAL, c);
    sagips_param_set ps;
    memset(&ps, 0, sizeof(ps));
    ps.n_tensors = 2;
    for (int i = 0; i < 2; ++i) {
      ps.param[i] = dev(2000 + 4 * i); ps.grad[i] = dev(2001 + 4 * i);
      ps.m[i] = dev(2002 + 4 * i); ps.v[i] = dev(2003 + 4 * i); ps.size[i] = 50049;
    }
    expect("adam ok", sagips_adam_step(c, &ps, 1, 1e-4, 0.9, 0.999, 1e-8), OK, c);
    expect("adam set NULL", sagips_adam_step(c, nullptr, 1, 1e-4, 0.9, 0.999, 1e-8), INVAL, c);
    expect("adam step 0", sagips_adam_step(c, &ps, 0, 1e-4, 0.9, 0.999, 1e-8), INVAL, c);
    expect("adam lr < 0", sagips_adam_step(c, &ps, 1, -1.0, 0.9, 0.999, 1e-8), INVAL, c);
    expect("adam beta1 = 1", sagips_adam_step(c, &ps, 1, 1e-4, 1.0, 0.999, 1e-8), INVAL, c);
    sagips_param_set q = ps; q.n_tensors = 17;
    expect("adam 17 tensors", sagips_adam_step(c, &q, 1, 1e-4, 0.9, 0.999, 1e-8), INVAL, c);
    q = ps; q.m[1] = nullptr;
    expect("adam m NULL", sagips_adam_step(c, &q, 1, 1e-4, 0.9, 0.999, 1e-8), INVAL, c);
    q = ps; q.size[0] = -1;
    expect("adam size < 0", sagips_adam_step(c, &q, 1, 1e-4, 0.9, 0.999, 1e-8), INVAL, c);
  }

  // ---- timing and streams
  {
    expect("set_timing on", sagips_set_timing(c, 1), OK, c);
    sagips_source s = source(4, 2, 1000);
    expect("timed sample", sagips_sample_events(c, &s, dev(1000), nullptr), OK, c);
    const char* names[8] = {};
    int64_t n[8] = {};
    double ms[8] = {};
    const int k = sagips_kernel_times(c, names, n, ms, 8);
    ++g_checks;
    if (k < 1 || !names[0] || n[0] < 1) { ++g_fail; printf("FAIL kernel_times returned %d\n", k); }
    expect("set_timing off", sagips_set_timing(c, 0), OK, c);
    expect("set_stream", sagips_set_stream(c, reinterpret_cast<void*>(0x1000)), OK, c);
    expect("set_stream back", sagips_set_stream(c, nullptr), OK, c);
  }
  expect("destroy", sagips_destroy(c), OK, nullptr);

  ++g_checks;
  if (stub_bad_launches() != 0) { ++g_fail; printf("FAIL %ld launches with a bad shape\n", stub_bad_launches()); }
  ++g_checks;
  if (stub_live_events() != 0) { ++g_fail; printf("FAIL %ld HIP events not destroyed\n", stub_live_events()); }
  ++g_checks;
  if (stub_live_allocs() != 0) { ++g_fail; printf("FAIL %ld device allocations not freed\n", stub_live_allocs()); }
  printf("%d checks, %d failed, %ld launches\n", g_checks, g_fail, stub_launches());
  if (g_fail == 0) printf("ALL OK\n");
  return g_fail == 0 ? 0 : 1;
}
