// A C-ABI caller with no Python: reads one decision step's inputs from a
// binary file, runs asymspec_fuse_verify on the current HIP device and
// writes the outputs.  Shows the calling sequence a serving engine uses:
// size and allocate the workspace once, upload, enqueue, synchronise.
//
// Input file (little endian): int32 B, K, V, dtype; then t, a, b
// [B][K+1][V] (2 or 4 bytes per logit), int32 drafts [B][K], float
// draft_probs [B][K], float uniforms [B][K+1], float temperature [B].
// Output file: int32 accept_len [B], int32 next_token [B], float
// fused_logprobs [B][K+1], float gate [B][K][2].
//
// Usage: fuse_verify_c <in> <out>

#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "asymspec.h"

#define CHECK_HIP(x)                                                          \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      std::fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));           \
      return 2;                                                               \
    }                                                                         \
  } while (0)

template <class T>
static bool read_n(std::FILE* f, std::vector<T>& v, size_t n) {
  v.resize(n);
  return std::fread(v.data(), sizeof(T), n, f) == n;
}

template <class T>
static int upload(const std::vector<T>& h, void** d) {
  CHECK_HIP(hipMalloc(d, h.size() * sizeof(T) + 16));
  CHECK_HIP(hipMemcpy(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice));
  return 0;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: %s <in> <out>\n", argv[0]);
    return 1;
  }
  std::FILE* f = std::fopen(argv[1], "rb");
  if (!f) return 1;
  int hdr[4];
  if (std::fread(hdr, sizeof(int), 4, f) != 4) return 1;
  const int B = hdr[0], K = hdr[1], V = hdr[2], dtype = hdr[3];
  const size_t nl = (size_t)B * (K + 1) * V, es = dtype == ASYMSPEC_BF16 ? 2 : 4;
  std::vector<unsigned char> t, a, b;
  std::vector<int> d;
  std::vector<float> q, u, tau;
  if (!read_n(f, t, nl * es) || !read_n(f, a, nl * es) || !read_n(f, b, nl * es) ||
      !read_n(f, d, (size_t)B * K) || !read_n(f, q, (size_t)B * K) ||
      !read_n(f, u, (size_t)B * (K + 1)) || !read_n(f, tau, (size_t)B))
    return 1;
  std::fclose(f);

  void *dt, *da, *db, *dd, *dq, *du, *dtau, *acc, *nxt, *flp, *gate, *ws;
  if (upload(t, &dt) || upload(a, &da) || upload(b, &db) || upload(d, &dd) || upload(q, &dq) ||
      upload(u, &du) || upload(tau, &dtau))
    return 2;
  CHECK_HIP(hipMalloc(&acc, B * sizeof(int)));
  CHECK_HIP(hipMalloc(&nxt, B * sizeof(int)));
  CHECK_HIP(hipMalloc(&flp, (size_t)B * (K + 1) * sizeof(float)));
  CHECK_HIP(hipMalloc(&gate, (size_t)B * (K > 0 ? K : 1) * 2 * sizeof(float)));
  const size_t wsb = asymspec_workspace_size(B, K, V, dtype);
  if (wsb == 0) return 3;
  CHECK_HIP(hipMalloc(&ws, wsb));

  asymspec_params p = {};
  p.beta = 1.0f;
  p.gamma = 0.5f;
  p.gate_mode = ASYMSPEC_GATE_CDA;
  p.delta_mode = ASYMSPEC_DELTA_AB;
  p.lambda = 0.1f;
  hipStream_t s;
  CHECK_HIP(hipStreamCreate(&s));
  const int st = asymspec_fuse_verify(dt, da, db, dtype, (const int32_t*)dd, (const float*)dq,
                                      (const float*)du, (const float*)dtau, B, K, V, &p, (int32_t*)acc,
                                      (int32_t*)nxt, (float*)flp, (float*)gate, nullptr, ws, wsb, s);
  if (st != ASYMSPEC_OK) {
    std::fprintf(stderr, "asymspec_fuse_verify: %s\n", asymspec_status_string(st));
    return 4;
  }
  CHECK_HIP(hipStreamSynchronize(s));

  std::vector<int> hacc(B), hnxt(B);
  std::vector<float> hflp((size_t)B * (K + 1)), hgate((size_t)B * K * 2);
  CHECK_HIP(hipMemcpy(hacc.data(), acc, B * sizeof(int), hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hnxt.data(), nxt, B * sizeof(int), hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(hflp.data(), flp, hflp.size() * sizeof(float), hipMemcpyDeviceToHost));
  if (K > 0) CHECK_HIP(hipMemcpy(hgate.data(), gate, hgate.size() * sizeof(float), hipMemcpyDeviceToHost));
  std::FILE* o = std::fopen(argv[2], "wb");
  if (!o) return 1;
  std::fwrite(hacc.data(), sizeof(int), B, o);
  std::fwrite(hnxt.data(), sizeof(int), B, o);
  std::fwrite(hflp.data(), sizeof(float), hflp.size(), o);
  std::fwrite(hgate.data(), sizeof(float), hgate.size(), o);
  std::fclose(o);
  for (void* x : {dt, da, db, dd, dq, du, dtau, acc, nxt, flp, gate, ws}) CHECK_HIP(hipFree(x));
  CHECK_HIP(hipStreamDestroy(s));
  std::printf("ok B=%d K=%d V=%d\n", B, K, V);
  return 0;
}
