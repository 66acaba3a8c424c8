// Native driver of the C ABI: runs a stored workload (one full encode, then
// incremental steps) with nothing but the HIP runtime and libincvit, so that
// hardware-counter passes can profile it without a Python runtime in the
// process.  Also does a plain device-to-device copy of known size, the
// calibration for the memory counters.
//
//   incvit_drive <dir> <steps> [full]  dir holds config.txt, weights.bin, frames.bin;
//                                     full: further full encodes of frame 0 after the first
//   incvit_drive --copy <MiB>
//
// config.txt: "img_h img_w channels patch dim depth heads mlp_dim dtype ln_eps
// views frames tau" then one cap per view.  weights.bin: canonical weights in
// the storage dtype.  frames.bin: float32 [frames][views][N][P].
// Prints one JSON line: steps, rows refreshed per step, launches per kernel kind.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "incvit.h"

namespace {

#define CHECK_HIP(x)                                                               \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));               \
      exit(3);                                                                     \
    }                                                                              \
  } while (0)
#define CHECK_IV(x, h)                                                             \
  do {                                                                             \
    incvit_status s_ = (x);                                                        \
    if (s_ != INCVIT_OK) {                                                         \
      fprintf(stderr, "%s failed (%d): %s\n", #x, (int)s_, incvit_last_error(h));  \
      exit(4);                                                                     \
    }                                                                              \
  } while (0)

std::vector<char> read_file(const std::string& path) {
  FILE* f = fopen(path.c_str(), "rb");
  if (!f) {
    fprintf(stderr, "cannot open %s\n", path.c_str());
    exit(2);
  }
  fseek(f, 0, SEEK_END);
  const long n = ftell(f);
  fseek(f, 0, SEEK_SET);
  std::vector<char> buf((size_t)n);
  if (n > 0 && fread(buf.data(), 1, (size_t)n, f) != (size_t)n) {
    fprintf(stderr, "short read of %s\n", path.c_str());
    exit(2);
  }
  fclose(f);
  return buf;
}

__global__ void copy_kernel(const uint4* src, uint4* dst, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

int copy_mode(int mib) {
  const size_t bytes = (size_t)mib << 20;
  void *a = nullptr, *b = nullptr;
  CHECK_HIP(hipMalloc(&a, bytes));
  CHECK_HIP(hipMalloc(&b, bytes));
  CHECK_HIP(hipMemset(a, 7, bytes));
  CHECK_HIP(hipDeviceSynchronize());
  const size_t n = bytes / 16;
  for (int r = 0; r < 3; ++r)
    hipLaunchKernelGGL(copy_kernel, dim3(2048), dim3(256), 0, 0, (const uint4*)a, (uint4*)b, n);
  CHECK_HIP(hipGetLastError());
  CHECK_HIP(hipDeviceSynchronize());
  printf("{\"copy_bytes\": %zu, \"reps\": 3, \"kernel\": \"copy_kernel\"}\n", bytes);
  CHECK_HIP(hipFree(a));
  CHECK_HIP(hipFree(b));
  return 0;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc == 3 && std::string(argv[1]) == "--copy") return copy_mode(atoi(argv[2]));
  if (argc < 3 || argc > 5) {
    fprintf(stderr, "usage: incvit_drive <dir> <steps> [full] [attn_qtiles] | incvit_drive --copy <MiB>\n");
    return 2;
  }
  const std::string dir = argv[1];
  const int steps = atoi(argv[2]);
  const int full_more = argc > 3 ? atoi(argv[3]) : 0;
  if (full_more < 0 || full_more > 1000) {
    fprintf(stderr, "full must be in [0, 1000]\n");
    return 2;
  }
  // query tiles per attention workgroup (0 = the library's choice)
  const int qtiles = argc > 4 ? atoi(argv[4]) : 0;
  if (qtiles < 0 || qtiles > 2) {
    fprintf(stderr, "attn_qtiles must be 0, 1 or 2\n");
    return 2;
  }

  incvit_config cfg;
  memset(&cfg, 0, sizeof cfg);
  int views = 0, frames = 0;
  float tau = 0.0f;
  std::vector<int32_t> caps;
  {
    std::vector<char> txt = read_file(dir + "/config.txt");
    txt.push_back(0);
    char* p = txt.data();
    char* end = nullptr;
    auto next = [&]() {
      const double v = strtod(p, &end);
      if (end == p) {
        fprintf(stderr, "bad config.txt\n");
        exit(2);
      }
      p = end;
      return v;
    };
    cfg.img_h = (int)next(); cfg.img_w = (int)next(); cfg.channels = (int)next(); cfg.patch = (int)next();
    cfg.dim = (int)next(); cfg.depth = (int)next(); cfg.heads = (int)next(); cfg.mlp_dim = (int)next();
    cfg.dtype = (int)next(); cfg.ln_eps = (float)next();
    views = (int)next(); frames = (int)next();
    tau = (float)next();
    for (int v = 0; v < views; ++v) caps.push_back((int32_t)next());
    cfg.max_streams = views;
  }
  if (steps < 0 || steps + 1 > frames) {
    fprintf(stderr, "need steps + 1 <= frames (%d)\n", frames);
    return 2;
  }
  const int N = (cfg.img_h / cfg.patch) * (cfg.img_w / cfg.patch);
  const int P = cfg.channels * cfg.patch * cfg.patch;
  const size_t eb = cfg.dtype == INCVIT_BF16 ? 2 : 4;

  std::vector<char> w = read_file(dir + "/weights.bin");
  if (w.size() != incvit_canonical_weights_bytes(&cfg)) {
    fprintf(stderr, "weights.bin has %zu bytes, expected %zu\n", w.size(), incvit_canonical_weights_bytes(&cfg));
    return 2;
  }
  std::vector<char> fr = read_file(dir + "/frames.bin");
  const size_t frame_bytes = (size_t)views * N * P * sizeof(float);
  if (fr.size() != frame_bytes * frames) {
    fprintf(stderr, "frames.bin has %zu bytes, expected %zu\n", fr.size(), frame_bytes * frames);
    return 2;
  }

  void *canon = nullptr, *packed = nullptr, *frames_d = nullptr, *ws = nullptr, *cache_buf = nullptr;
  void *idx = nullptr, *count = nullptr, *refreshed = nullptr;
  CHECK_HIP(hipMalloc(&canon, w.size()));
  CHECK_HIP(hipMemcpy(canon, w.data(), w.size(), hipMemcpyHostToDevice));
  const size_t pbytes = incvit_packed_weights_bytes(&cfg);
  CHECK_HIP(hipMalloc(&packed, pbytes));
  CHECK_IV(incvit_pack_weights(&cfg, canon, packed, nullptr), nullptr);
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipFree(canon));
  incvit_handle* h = nullptr;
  CHECK_IV(incvit_create(&cfg, packed, &h), nullptr);
  if (qtiles) {
    incvit_tuning t;
    memset(&t, 0, sizeof t);
    t.attn_qtiles = qtiles;
    CHECK_IV(incvit_set_tuning(h, &t), h);
  }

  CHECK_HIP(hipMalloc(&frames_d, fr.size()));
  CHECK_HIP(hipMemcpy(frames_d, fr.data(), fr.size(), hipMemcpyHostToDevice));
  const size_t cbytes = incvit_cache_bytes(h);
  CHECK_HIP(hipMalloc(&cache_buf, cbytes * views));
  CHECK_HIP(hipMemset(cache_buf, 0, cbytes * views));
  std::vector<void*> caches(views);
  for (int v = 0; v < views; ++v) caches[v] = static_cast<char*>(cache_buf) + cbytes * v;
  CHECK_HIP(hipMalloc(&ws, incvit_workspace_bytes(h, views)));
  CHECK_HIP(hipMalloc(&idx, (size_t)views * N * 4));
  CHECK_HIP(hipMalloc(&count, (size_t)views * 4));
  CHECK_HIP(hipMalloc(&refreshed, (size_t)views * N * cfg.dim * eb));

  auto frame = [&](int t) { return reinterpret_cast<const float*>(static_cast<char*>(frames_d) + frame_bytes * t); };
  CHECK_IV(incvit_full_encode(h, views, frame(0), caches.data(), ws, nullptr), h);
  for (int r = 0; r < full_more; ++r) CHECK_IV(incvit_full_encode(h, views, frame(0), caches.data(), ws, nullptr), h);
  std::vector<int32_t> cnt(views);
  std::vector<long> rows;
  for (int t = 1; t <= steps; ++t) {
    CHECK_IV(incvit_step(h, views, frame(t), caches.data(), tau, caps.data(), (int32_t*)idx, (int32_t*)count,
                         refreshed, ws, nullptr), h);
    CHECK_HIP(hipMemcpy(cnt.data(), count, (size_t)views * 4, hipMemcpyDeviceToHost));
    long m = 0;
    for (int v = 0; v < views; ++v) m += cnt[v];
    rows.push_back(m);
  }
  CHECK_HIP(hipDeviceSynchronize());
  for (int v = 0; v < views; ++v) {
    const incvit_status st = incvit_cache_status(h, caches[v], nullptr);
    if (st != INCVIT_OK) {
      fprintf(stderr, "stream %d: cache status %d\n", v, (int)st);
      return 5;
    }
  }
  // launches of the timed steps per kernel kind (steps with no refreshed row
  // launch only the selection kernels)
  long capsum = 0;
  for (int32_t c : caps) capsum += std::min(std::max(c, 0), N);
  const long active = capsum > 0 ? steps : 0;  // a step with caps > 0 launches every kernel
  double mean = 0.0;
  for (long m : rows) mean += (double)m / (rows.empty() ? 1 : rows.size());
  const long L = cfg.depth;
  printf("{\"steps\": %d, \"rows_mean\": %.3f, \"kernel_launches\": {\"embed\": %d, \"sim\": %d, \"select\": %d, "
         "\"commit\": %ld, \"qkv\": %ld, \"attn\": %ld, \"oproj\": %ld, \"fc1\": %ld, \"fc2\": %ld, "
         "\"res_ln1\": %ld}, \"full_encodes\": %d, \"views\": %d, \"tokens\": %d, \"dim\": %d, \"depth\": %d, "
         "\"mlp\": %d, \"config\": {\"workload\": \"%s\", \"rows_mean\": %.3f}}\n",
         steps, mean, steps, steps, steps, active, active * L, active * L, active * L, active * L, active * L,
         active * L, full_more + 1, views, N, cfg.dim, cfg.depth, cfg.mlp_dim, dir.c_str(), mean);
  incvit_destroy(h);
  return 0;
}
