// Drives every host-only path of libhapi (descriptor validation, shape and
// byte calculus, workspace layout, profiles without timing, split choice and
// their error paths) under AddressSanitizer and UBSan.  Model descriptors are
// read from a text file the test writes from the Python model definitions:
//   model <dtype> <in_c> <in_h> <in_w> <n_layers>
//   <kind> <cin> <cout> <width> <k> <stride> <pad> <relu> <has_bias> <has_bn> <heads> <mlp_dim>
// Buffers are heap blocks of exactly the size each entry point may write, so
// any write past them is reported.  Prints "OK <calls>" on success.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "hapi.h"

static long g_calls = 0;
#define EXPECT(cond)                                                       \
  do {                                                                     \
    ++g_calls;                                                             \
    if (!(cond)) {                                                         \
      std::fprintf(stderr, "FAILED %s at line %d: %s\n", #cond, __LINE__, hapi_last_error()); \
      std::exit(2);                                                        \
    }                                                                      \
  } while (0)

template <class T>
static T *exact(size_t n) {  // n elements, nothing more (n >= 1)
  return static_cast<T *>(std::malloc(sizeof(T) * (n ? n : 1)));
}

static void exercise(hapi_model_desc d) {
  const int n = d.n_layers;
  EXPECT(hapi_raw_weight_count(&d) >= 0);
  EXPECT(hapi_packed_weight_bytes(&d) >= 0);
  for (int k = 0; k <= n; ++k) {
    int64_t *dims = exact<int64_t>(3);
    int32_t *nd = exact<int32_t>(1);
    EXPECT(hapi_layer_shape(&d, k, dims, nd) == HAPI_OK && (*nd == 2 || *nd == 3));
    std::free(dims);
    std::free(nd);
  }
  const int batches[] = {1, 3, 64, 128, 257};
  const int chunks[] = {0, 1, 7, 64};
  for (int b : batches)
    for (int c : chunks)
      for (int inf = 0; inf <= 4; ++inf) {
        hapi_model_desc e = d;
        e.chunk = c;
        e.inflight = inf;
        EXPECT(hapi_chunk_count(&e, b) >= 1);
        for (int s = 0; s <= n; s += (n > 6 ? 3 : 1)) {
          EXPECT(hapi_workspace_bytes(&e, b, s, 0) >= 0);
          EXPECT(hapi_workspace_bytes(&e, b, s, 1) >= 0);
          const int g = hapi_workspace_guards(&e, b, s, nullptr, 0);
          EXPECT(g >= 0);
          int64_t *off = exact<int64_t>(g);
          EXPECT(hapi_workspace_guards(&e, b, s, off, g) == g);
          std::free(off);
        }
        int64_t *bytes = exact<int64_t>(n + 1);
        EXPECT(hapi_profile_layers(&e, b, bytes, nullptr) == HAPI_OK);
        EXPECT(hapi_profile_memory(&e, b, bytes) == HAPI_OK);
        std::free(bytes);
      }
  // error paths: each fails validation and writes nothing
  int64_t dims[3];
  int32_t nd;
  EXPECT(hapi_layer_shape(&d, -1, dims, &nd) == HAPI_E_INVAL);
  EXPECT(hapi_layer_shape(&d, n + 1, dims, &nd) == HAPI_E_INVAL);
  EXPECT(hapi_workspace_bytes(&d, 0, n, 0) == HAPI_E_INVAL);
  EXPECT(hapi_workspace_bytes(&d, 2, n + 1, 0) == HAPI_E_INVAL);
  EXPECT(hapi_workspace_guards(&d, 2, -1, nullptr, 0) == HAPI_E_INVAL);
  hapi_model_desc e = d;
  e.inflight = 5;
  EXPECT(hapi_chunk_count(&e, 4) == HAPI_E_INVAL);
  e = d;
  e.direct = 2;
  EXPECT(hapi_chunk_count(&e, 4) == HAPI_E_INVAL);
  e = d;
  e.dtype = 7;
  EXPECT(hapi_raw_weight_count(&e) == HAPI_E_INVAL);
  // extraction without a workspace: refused before any launch
  alignas(256) static char dummy[1024];
  e = d;
  e.workspace = nullptr;
  e.workspace_bytes = 0;
  EXPECT(hapi_extract(&e, dummy, dummy, 2, n, dummy) == HAPI_E_NOMEM);
  EXPECT(hapi_extract(&e, dummy, nullptr, 2, n, dummy) == HAPI_E_INVAL);
  EXPECT(hapi_extract_range(&e, dummy, dummy, 2, n, n - 1, dummy) == HAPI_E_INVAL);
  EXPECT(std::strlen(hapi_last_error()) > 0);
  // a reserved field set
  std::vector<hapi_layer> bad(d.layers, d.layers + n);
  bad[n - 1].reserved[2] = 1;
  e = d;
  e.layers = bad.data();
  EXPECT(hapi_packed_weight_bytes(&e) == HAPI_E_INVAL);

  // split choice over this model's per-image output bytes
  int64_t *img = exact<int64_t>(n + 1);
  EXPECT(hapi_profile_layers(&d, 1, img, nullptr) == HAPI_OK);
  double *srv = exact<double>(n + 1), *cli = exact<double>(n + 1);
  for (int k = 0; k <= n; ++k) {
    srv[k] = k ? 1e-3 * (1 + k % 3) : 0.0;
    cli[k] = k ? 2e-3 * (1 + k % 2) : 0.0;
  }
  hapi_split_job j;
  std::memset(&j, 0, sizeof j);
  j.n_layers = n;
  j.freeze_idx = n - 1;
  j.train_batch = 512;
  j.request_images = 128;
  j.server_slots = 4;
  j.iterations = 60;
  j.image_bytes = img;
  j.srv_layer_s = srv;
  j.cli_layer_s = cli;
  j.srv_read_data_s = 0.05;
  j.srv_read_model_s = 0.1;
  j.srv_to_gpu_s = 0.01;
  j.cli_rest_s = 0.2;
  j.srv_from_gpu_s_per_byte = 1e-10;
  j.srv_pickle_s_per_byte = 5e-10;
  j.cli_unpickle_s_per_byte = 5e-10;
  j.cli_loader_s_per_byte = 2e-10;
  j.cli_to_gpu_s_per_byte = 1e-10;
  j.net_bytes_per_s = 1.5e9;
  hapi_split_estimate *est = exact<hapi_split_estimate>(j.freeze_idx + 1);
  hapi_split_choice ch;
  EXPECT(hapi_choose_split(&j, est, &ch) == HAPI_OK);
  EXPECT(ch.hapi >= 0 && ch.hapi <= j.freeze_idx);
  j.cli_mem_bytes = 1;  // even the freeze split cannot fit
  EXPECT(hapi_choose_split(&j, est, &ch) == HAPI_E_NOMEM);
  j.cli_mem_bytes = 0;
  j.train_batch = 500;  // not a multiple of the request size
  EXPECT(hapi_choose_split(&j, est, &ch) == HAPI_E_INVAL);
  std::free(est);
  std::free(img);
  std::free(srv);
  std::free(cli);
}

int main(int argc, char **argv) {
  if (argc != 2) return 1;
  FILE *f = std::fopen(argv[1], "r");
  if (!f) return 1;
  char tag[32];
  int models = 0;
  while (std::fscanf(f, "%31s", tag) == 1) {
    hapi_model_desc d;
    std::memset(&d, 0, sizeof d);
    int n = 0;
    if (std::strcmp(tag, "model") != 0 ||
        std::fscanf(f, "%d %d %d %d %d", &d.dtype, &d.in_c, &d.in_h, &d.in_w, &n) != 5)
      return 1;
    std::vector<hapi_layer> L(n);
    for (int i = 0; i < n; ++i) {
      hapi_layer &l = L[i];
      std::memset(&l, 0, sizeof l);
      if (std::fscanf(f, "%d %d %d %d %d %d %d %d %d %d %d %d", &l.kind, &l.cin, &l.cout, &l.width, &l.k,
                      &l.stride, &l.pad, &l.relu, &l.has_bias, &l.has_bn, &l.heads, &l.mlp_dim) != 12)
        return 1;
    }
    d.n_layers = n;
    d.layers = L.data();
    exercise(d);
    ++models;
  }
  std::fclose(f);
  EXPECT(hapi_raw_weight_count(nullptr) == HAPI_E_INVAL);
  std::printf("OK %d models, %ld checks\n", models, g_calls);
  return 0;
}
