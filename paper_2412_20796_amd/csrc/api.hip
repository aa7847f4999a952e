// C-ABI entry points, hyperparameter validation and the flat parameter layout.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <map>
#include <string>
#include <vector>

#include "common.hpp"

namespace chg {

size_t graph_scratch_bytes(int64_t N, int64_t S);
size_t acts_bytes(const chgnet_hparams& hp, int64_t N, int64_t E, int64_t B, int64_t A, int64_t S);
int build_graph(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws, size_t ws_bytes,
                hipStream_t st);
int build_graph_noalloc(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, hipStream_t st);
int forward_entry(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                  float* energy, float* forces, float* stress, float* magmom, int save_for_backward, void* ws,
                  size_t ws_bytes, hipStream_t st);
int backward_entry(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                   const float* dE, const float* dF, const float* dS, const float* dM, float* grad, void* ws,
                   size_t ws_bytes, hipStream_t st);
int step_entry(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, float* params,
               const float* E_t, const float* F_t, const float* S_t, const float* M_t, const chgnet_loss* loss_cfg,
               float* loss, float* grad, float* adam_m, float* adam_v, const float* adam_hp, void* ws,
               size_t ws_bytes, hipStream_t st);
int md_entry(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, const float* params,
             chgnet_md_state* s, float dt, int n_steps, int forces_valid, int* steps_done, void* ws,
             size_t ws_bytes, hipStream_t st);

namespace {
thread_local std::string g_last_error;

// Per-launch event timing for measurement (chgnet_profile_start/stop).
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> ev;
  size_t used = 0;
  struct Rec { std::string tag; int a, b; };
  std::vector<Rec> recs;
};
Profiler g_prof;
}  // namespace

int prof_mark(hipStream_t st) {
  if (!g_prof.on || g_prof.used + 2 > g_prof.ev.size()) return -1;
  const int i = (int)g_prof.used;
  if (hipEventRecord(g_prof.ev[i], st) != hipSuccess) return -1;
  g_prof.used += 2;
  return i;
}

bool prof_active() { return g_prof.on; }

void prof_close(hipStream_t st, int first, const char* tag) {
  if (first < 0) return;
  (void)hipEventRecord(g_prof.ev[first + 1], st);
  g_prof.recs.push_back({tag, first, first + 1});
}

void set_error(const std::string& msg) { g_last_error = msg; }
int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int validate_hparams(const chgnet_hparams* hp) {
  if (!hp) return fail(CHGNET_EINVAL, "hparams is NULL");
  if (hp->d != 64 && hp->d != 128) return fail(CHGNET_EINVAL, "d must be 64 or 128");
  if (hp->n_layers < 1 || hp->n_layers > kMaxLayers) return fail(CHGNET_EINVAL, "n_layers must be in 1..16");
  if (hp->n_rbf < 1 || hp->n_rbf > 64) return fail(CHGNET_EINVAL, "n_rbf must be in 1..64");
  if (hp->n_fourier < 1 || hp->n_fourier > 63 || hp->n_fourier % 2 == 0)
    return fail(CHGNET_EINVAL, "n_fourier must be odd and in 1..63");
  if (hp->envelope_p < 2 || hp->envelope_p > 16) return fail(CHGNET_EINVAL, "envelope_p must be in 2..16");
  if (!(hp->r_bond > 0.f) || !(hp->r_bond <= hp->r_atom) || !(hp->r_atom <= 20.f))
    return fail(CHGNET_EINVAL, "cutoffs must satisfy 0 < r_bond <= r_atom <= 20");
  if ((hp->magmom != 0 && hp->magmom != 1) || (hp->sequential != 0 && hp->sequential != 1) ||
      (hp->conservative != 0 && hp->conservative != 1))
    return fail(CHGNET_EINVAL, "magmom, sequential and conservative must be 0 or 1");
  return CHGNET_OK;
}

ParamLayout make_layout(const chgnet_hparams& hp, int align) {
  ParamLayout L{};
  const int64_t d = hp.d, R = hp.n_rbf, K = hp.n_fourier;
  int64_t off = 0;
  auto take = [&](int64_t n) {
    off = (off + align - 1) / align * align;
    int64_t o = off;
    off += n;
    L.toff[L.ntensors] = o;
    L.tlen[L.ntensors] = n;
    L.ntensors++;
    return o;
  };
  L.W_Z = take(94 * d);
  L.f_a = take(R);
  L.f_b = take(R);
  L.W_e = take(R * 2 * d);
  L.b_e0 = take(d);
  L.W_eb = take(R * d);
  L.W_th = take(K * d);
  L.b_th = take(d);
  auto gated = [&](int64_t rows) {
    GatedOffsets g;
    g.W = take(rows * 2 * d);
    g.b = take(2 * d);
    g.g_c = take(d);
    g.b_c = take(d);
    g.g_g = take(d);
    g.b_g = take(d);
    return g;
  };
  for (int t = 0; t < hp.n_layers; ++t) {
    LayerOffsets& lo = L.layer[t];
    lo.av = gated(3 * d);
    lo.av_Wo = take(d * d);
    lo.av_bo = take(d);
    lo.be = gated(4 * d);
    lo.be_Wo = take(d * d);
    lo.be_bo = take(d);
    lo.has_angle = t < hp.n_layers - 1;
    if (lo.has_angle) lo.an = gated(4 * d);
    else lo.an = lo.be;
  }
  const int outs[3] = {1, 1, 9};
  for (int h = 0; h < 3; ++h) {
    HeadOffsets& ho = L.head[h];
    ho.out = outs[h];
    ho.W1 = take(d * d);
    ho.b1 = take(d);
    ho.W2 = take(d * d);
    ho.b2 = take(d);
    ho.W3 = take(d * ho.out);
    ho.b3 = take(ho.out);
  }
  L.M_W = L.M_b = -1;
  if (hp.magmom) {
    L.M_W = take(d);
    L.M_b = take(1);
  }
  L.total = off;
  return L;
}

}  // namespace chg

extern "C" {

int chgnet_param_count(const chgnet_hparams* hp, int64_t* n) {
  CHG_TRY(chg::validate_hparams(hp));
  if (!n) return chg::fail(CHGNET_EINVAL, "n is NULL");
  *n = chg::make_layout(*hp).total;
  return CHGNET_OK;
}

int chgnet_workspace_size(const chgnet_hparams* hp, int64_t N, int64_t E, int64_t B, int64_t A, int64_t S,
                          size_t* bytes) {
  CHG_TRY(chg::validate_hparams(hp));
  if (!bytes || N < 0 || E < 0 || B < 0 || A < 0 || S < 0) return chg::fail(CHGNET_EINVAL, "bad sizes");
  *bytes = chg::graph_scratch_bytes(N, S) + chg::acts_bytes(*hp, N, E, B, A, S);
  return CHGNET_OK;
}

int chgnet_build_graph(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, void* ws,
                       size_t ws_bytes, void* stream) {
  return chg::build_graph(hp, batch, graph, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int chgnet_build_graph_noalloc(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph,
                               void* stream) {
  return chg::build_graph_noalloc(hp, batch, graph, static_cast<hipStream_t>(stream));
}

int chgnet_forward(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                   float* energy, float* forces, float* stress, float* magmom, int save_for_backward, void* ws,
                   size_t ws_bytes, void* stream) {
  return chg::forward_entry(hp, batch, graph, params, energy, forces, stress, magmom, save_for_backward, ws, ws_bytes,
                            static_cast<hipStream_t>(stream));
}

int chgnet_backward(const chgnet_hparams* hp, const chgnet_batch* batch, const chgnet_graph* graph, const float* params,
                    const float* dE, const float* dF, const float* dS, const float* dM, float* grad, void* ws,
                    size_t ws_bytes, void* stream) {
  return chg::backward_entry(hp, batch, graph, params, dE, dF, dS, dM, grad, ws, ws_bytes,
                             static_cast<hipStream_t>(stream));
}

int chgnet_step(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, float* params,
                const float* E_target, const float* F_target, const float* S_target, const float* M_target,
                const chgnet_loss* loss_cfg, float* loss, float* grad, float* adam_m, float* adam_v,
                const float* adam_hp, void* ws, size_t ws_bytes, void* stream) {
  return chg::step_entry(hp, batch, graph, params, E_target, F_target, S_target, M_target, loss_cfg, loss, grad,
                         adam_m, adam_v, adam_hp, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int chgnet_md(const chgnet_hparams* hp, const chgnet_batch* batch, chgnet_graph* graph, const float* params,
              chgnet_md_state* state, float dt, int n_steps, int forces_valid, int* steps_done, void* ws,
              size_t ws_bytes, void* stream) {
  return chg::md_entry(hp, batch, graph, params, state, dt, n_steps, forces_valid, steps_done, ws, ws_bytes,
                       static_cast<hipStream_t>(stream));
}

const char* chgnet_last_error_string(void) { return chg::g_last_error.c_str(); }

int chgnet_profile_start(int max_launches) {
  auto& P = chg::g_prof;
  if (max_launches < 1) return chg::fail(CHGNET_EINVAL, "max_launches must be >= 1");
  while ((int)P.ev.size() < 2 * max_launches) {
    hipEvent_t e;
    CHG_HIP(hipEventCreate(&e));
    P.ev.push_back(e);
  }
  P.used = 0;
  P.recs.clear();
  P.on = true;
  return CHGNET_OK;
}

int chgnet_profile_stop(char* buf, size_t buflen) {
  auto& P = chg::g_prof;
  P.on = false;
  std::map<std::string, std::pair<int64_t, double>> agg;
  for (const auto& r : P.recs) {
    CHG_HIP(hipEventSynchronize(P.ev[r.b]));
    float ms = 0.f;
    CHG_HIP(hipEventElapsedTime(&ms, P.ev[r.a], P.ev[r.b]));
    auto& x = agg[r.tag];
    x.first += 1;
    x.second += ms;
  }
  std::string out;
  char line[256];
  for (const auto& kv : agg) {
    std::snprintf(line, sizeof(line), "%s %lld %.6f\n", kv.first.c_str(), (long long)kv.second.first, kv.second.second);
    out += line;
  }
  const bool truncated = P.used + 2 > P.ev.size();
  P.recs.clear();
  P.used = 0;
  if (!buf || buflen <= out.size()) return chg::fail(CHGNET_EINVAL, "profile buffer too small");
  std::snprintf(buf, buflen, "%s", out.c_str());
  return truncated ? chg::fail(CHGNET_EWORKSPACE, "more launches than max_launches; later ones not timed") : CHGNET_OK;
}

}  // extern "C"
