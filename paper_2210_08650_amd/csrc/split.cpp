// Split-index choice: the epoch-runtime model of Algorithm 1 over the
// per-layer profile, plus the static (NoSplit, @Freeze, @Min) and NSG
// competitors of the evaluation.  Host arithmetic only; the formulas are
// stated next to hapi_choose_split in hapi.h.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "internal.h"

namespace hapi {
namespace {

bool finite_nonneg(double v) { return std::isfinite(v) && v >= 0.0; }

// a * b for non-negative int64 values, false on overflow.
bool mul_ok(int64_t a, int64_t b, int64_t *r) {
  if (a != 0 && b > std::numeric_limits<int64_t>::max() / a) return false;
  *r = a * b;
  return true;
}

bool add_ok(int64_t a, int64_t b, int64_t *r) {
  if (b > std::numeric_limits<int64_t>::max() - a) return false;
  *r = a + b;
  return true;
}

int validate(const hapi_split_job *j, const hapi_split_choice *choice) {
  if (!j || !choice) return fail(HAPI_E_INVAL, "job and choice must not be NULL");
  if (j->n_layers < 1) return fail(HAPI_E_INVAL, "n_layers must be >= 1");
  if (j->freeze_idx < 0 || j->freeze_idx > j->n_layers)
    return fail(HAPI_E_INVAL, "freeze_idx %d outside [0, %d]", j->freeze_idx, j->n_layers);
  if (j->train_batch < 1 || j->request_images < 1 || j->server_slots < 1)
    return fail(HAPI_E_INVAL, "train_batch, request_images and server_slots must be >= 1");
  if (j->train_batch % j->request_images != 0)
    return fail(HAPI_E_INVAL, "train_batch %d is not a multiple of request_images %d",
                j->train_batch, j->request_images);
  if (j->reserved0 != 0) return fail(HAPI_E_INVAL, "reserved0 must be 0");
  if (j->iterations < 1) return fail(HAPI_E_INVAL, "iterations must be >= 1");
  if (!j->image_bytes || !j->srv_layer_s || !j->cli_layer_s)
    return fail(HAPI_E_INVAL, "image_bytes, srv_layer_s and cli_layer_s must not be NULL");
  for (int k = 0; k <= j->n_layers; ++k) {
    if (j->image_bytes[k] < 1) return fail(HAPI_E_INVAL, "image_bytes[%d] must be >= 1", k);
    if (k > 0 && (!finite_nonneg(j->srv_layer_s[k]) || !finite_nonneg(j->cli_layer_s[k])))
      return fail(HAPI_E_INVAL, "layer %d: times must be finite and >= 0", k);
  }
  const double phases[] = {j->srv_read_data_s,        j->srv_read_model_s,
                           j->srv_to_gpu_s,            j->cli_rest_s,
                           j->srv_from_gpu_s_per_byte, j->srv_pickle_s_per_byte,
                           j->cli_unpickle_s_per_byte, j->cli_loader_s_per_byte,
                           j->cli_to_gpu_s_per_byte};
  for (double v : phases)
    if (!finite_nonneg(v)) return fail(HAPI_E_INVAL, "phase times and rates must be finite and >= 0");
  if (!(std::isfinite(j->net_bytes_per_s) && j->net_bytes_per_s > 0.0))
    return fail(HAPI_E_INVAL, "net_bytes_per_s must be finite and > 0");
  if (!std::isfinite(j->nosplit_iter_s)) return fail(HAPI_E_INVAL, "nosplit_iter_s must be finite");
  if (j->cli_mem_bytes < 0 || j->cli_fixed_mem_bytes < 0)
    return fail(HAPI_E_INVAL, "memory sizes must be >= 0");
  return HAPI_OK;
}

}  // namespace
}  // namespace hapi

using namespace hapi;

extern "C" int hapi_choose_split(const hapi_split_job *j, hapi_split_estimate *est,
                                 hapi_split_choice *choice) {
  if (int st = validate(j, choice)) return st;
  const int n = j->n_layers, F = j->freeze_idx;
  const int64_t B = j->train_batch, R = j->request_images;
  const int64_t requests = B / R;
  const int64_t waves = (requests + j->server_slots - 1) / j->server_slots;

  // Client memory (largest input + output of the layers the client runs,
  // beside the received split output) for every split 0..n, computed from the
  // back: peak[s] = max(image_bytes[s], max_{k>s} in_k + out_k).
  std::vector<int64_t> peak(n + 1);
  int64_t tail = 0;
  for (int s = n; s >= 0; --s) {
    if (s < n) {
      int64_t io;
      if (!add_ok(j->image_bytes[s], j->image_bytes[s + 1], &io))
        return fail(HAPI_E_INVAL, "image_bytes overflow at layer %d", s + 1);
      tail = std::max(tail, io);
    }
    peak[s] = std::max(tail, j->image_bytes[s]);
  }

  std::vector<hapi_split_estimate> e(F + 1);
  double srv_fwd = 0.0;  // one request's forward time through layers 1..s
  const double linear_cli =
      j->cli_unpickle_s_per_byte + j->cli_loader_s_per_byte + j->cli_to_gpu_s_per_byte;
  for (int s = 0; s <= F; ++s) {
    if (s > 0) srv_fwd += j->srv_layer_s[s];
    double cli_fwd = 0.0;  // client forward time through layers s+1..n
    for (int k = s + 1; k <= n; ++k) cli_fwd += j->cli_layer_s[k];
    int64_t mem;
    if (!mul_ok(B, peak[s], &mem) || !add_ok(mem, j->cli_fixed_mem_bytes, &mem))
      return fail(HAPI_E_INVAL, "client memory estimate overflows at split %d", s);
    const double req_bytes = (double)R * (double)j->image_bytes[s];
    const double batch_bytes = (double)B * (double)j->image_bytes[s];
    hapi_split_estimate &x = e[s];
    x = hapi_split_estimate{};
    double per_wave = j->srv_read_data_s + req_bytes * j->srv_pickle_s_per_byte;
    if (s > 0)
      per_wave += j->srv_read_model_s + j->srv_to_gpu_s + req_bytes * j->srv_from_gpu_s_per_byte;
    x.rt_srv = (double)waves * per_wave + (double)requests * srv_fwd;
    x.rt_nw = batch_bytes / j->net_bytes_per_s;
    x.rt_cli = batch_bytes * linear_cli + cli_fwd + j->cli_rest_s;
    x.sum_s = x.rt_srv + x.rt_nw + x.rt_cli;
    if (s == 0 && j->nosplit_iter_s > 0.0)
      x.epoch_s = (double)j->iterations * j->nosplit_iter_s;
    else
      x.epoch_s = x.rt_srv + std::max(x.rt_srv + x.rt_nw, x.rt_cli) * (double)(j->iterations - 1) +
                  x.rt_cli;
    x.cli_mem_bytes = mem;
    x.oom = (j->cli_mem_bytes > 0 && mem > j->cli_mem_bytes) ? 1 : 0;
  }
  if (e[F].oom)
    return fail(HAPI_E_NOMEM,
                "the freeze split %d needs %lld client bytes (> %lld); every earlier split needs at least as much",
                F, (long long)e[F].cli_mem_bytes, (long long)j->cli_mem_bytes);

  hapi_split_choice c{};
  c.freeze = F;
  c.nosplit = 0;
  c.earliest = -1;
  c.hapi = c.nsg = -1;
  for (int s = 0; s <= F; ++s) {
    if (e[s].oom) continue;
    if (c.earliest < 0) c.earliest = s;
    if (c.hapi < 0 || e[s].epoch_s < e[c.hapi].epoch_s) c.hapi = s;
    if (c.nsg < 0 || e[s].sum_s < e[c.nsg].sum_s) c.nsg = s;
  }
  c.min_output = 0;
  for (int k = 1; k <= F; ++k)
    if (c.min_output == 0 || j->image_bytes[k] < j->image_bytes[c.min_output]) c.min_output = k;

  if (est)
    for (int s = 0; s <= F; ++s) est[s] = e[s];
  *choice = c;
  return HAPI_OK;
}
