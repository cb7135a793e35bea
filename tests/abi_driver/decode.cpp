// Decode attention through the C ABI alone (HIP runtime + halo_attn.h, no
// Python): reads one batch from a file, runs plan, upload and decode, and
// writes O and LSE to a file. Used by the GPU tests to check that the
// library is usable from C and C++ as declared.
//
// Input (little-endian): int32 num_q_heads, num_kv_heads, head_dim, kv_dtype,
// out_dtype, num_pool_pages, num_segments, num_requests; float sm_scale;
// int32 seg_len[S], seg_page_indptr[S+1], seg_page_ids[seg_page_indptr[S]],
// req_seg_indptr[R+1], req_seg_ids[req_seg_indptr[R]]; then the raw bytes
// of q [R][H_q][d], k_pool and v_pool [num_pool_pages][H_kv][16 d] (kv_dtype).
// Output: o [R][H_q][d] (out_dtype bytes), then lse [R][H_q] float32.
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "halo_attn.h"

namespace {

void die(const char* what) {
  std::fprintf(stderr, "error: %s\n", what);
  std::exit(1);
}

void hip_ok(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    std::exit(1);
  }
}

void halo_ok(halo_status_t s, const char* what) {
  if (s != HALO_OK) {
    std::fprintf(stderr, "%s: %s (%s)\n", what, halo_status_string(s), halo_last_error_message());
    std::exit(1);
  }
}

template <typename T>
std::vector<T> read_n(FILE* f, size_t n) {
  std::vector<T> v(n);
  if (n && std::fread(v.data(), sizeof(T), n, f) != n) die("short input");
  return v;
}

void* to_device(const std::vector<unsigned char>& h) {
  void* d = nullptr;
  hip_ok(hipMalloc(&d, h.size() ? h.size() : 16), "hipMalloc");
  if (h.size()) hip_ok(hipMemcpy(d, h.data(), h.size(), hipMemcpyHostToDevice), "hipMemcpy");
  return d;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) die("usage: decode INPUT OUTPUT");
  FILE* f = std::fopen(argv[1], "rb");
  if (!f) die("cannot open input");
  const std::vector<int32_t> hdr = read_n<int32_t>(f, 8);
  const float scale = read_n<float>(f, 1)[0];
  halo_attn_params_t p{};
  p.num_q_heads = hdr[0];
  p.num_kv_heads = hdr[1];
  p.head_dim = hdr[2];
  p.page_size = 16;
  p.num_pool_pages = hdr[5];
  p.kv_dtype = static_cast<halo_dtype_t>(hdr[3]);
  p.out_dtype = static_cast<halo_dtype_t>(hdr[4]);
  p.sm_scale = scale;
  const int S = hdr[6], R = hdr[7];
  const std::vector<int32_t> seg_len = read_n<int32_t>(f, S);
  const std::vector<int32_t> seg_page_indptr = read_n<int32_t>(f, S + 1);
  const std::vector<int32_t> seg_page_ids = read_n<int32_t>(f, seg_page_indptr[S]);
  const std::vector<int32_t> req_seg_indptr = read_n<int32_t>(f, R + 1);
  const std::vector<int32_t> req_seg_ids = read_n<int32_t>(f, req_seg_indptr[R]);
  const size_t elt = p.kv_dtype == HALO_BF16 ? 2 : 4;
  const size_t out_elt = p.out_dtype == HALO_BF16 ? 2 : 4;
  const size_t q_bytes = (size_t)R * p.num_q_heads * p.head_dim * elt;
  const size_t pool_bytes = (size_t)p.num_pool_pages * p.num_kv_heads * 16 * p.head_dim * elt;
  const std::vector<unsigned char> q = read_n<unsigned char>(f, q_bytes);
  const std::vector<unsigned char> kp = read_n<unsigned char>(f, pool_bytes);
  const std::vector<unsigned char> vp = read_n<unsigned char>(f, pool_bytes);
  std::fclose(f);

  halo_forest_t forest{};
  forest.num_segments = S;
  forest.seg_len = seg_len.data();
  forest.seg_page_indptr = seg_page_indptr.data();
  forest.seg_page_ids = seg_page_ids.data();
  forest.num_requests = R;
  forest.req_seg_indptr = req_seg_indptr.data();
  forest.req_seg_ids = req_seg_ids.data();
  forest.q_len = nullptr;

  halo_plan_t* plan = nullptr;
  size_t meta_bytes = 0, ws_bytes = 0;
  halo_ok(halo_plan_create(&p, &forest, &plan, &meta_bytes, &ws_bytes), "halo_plan_create");
  void *d_meta = nullptr, *d_ws = nullptr, *d_o = nullptr;
  float* d_lse = nullptr;
  hip_ok(hipMalloc(&d_meta, meta_bytes), "hipMalloc meta");
  if (ws_bytes) hip_ok(hipMalloc(&d_ws, ws_bytes), "hipMalloc workspace");
  const size_t rows = (size_t)R * p.num_q_heads;
  hip_ok(hipMalloc(&d_o, rows * p.head_dim * out_elt), "hipMalloc o");
  hip_ok(hipMalloc(reinterpret_cast<void**>(&d_lse), rows * sizeof(float)), "hipMalloc lse");
  void* d_q = to_device(q);
  void* d_k = to_device(kp);
  void* d_v = to_device(vp);
  hipStream_t stream;
  hip_ok(hipStreamCreate(&stream), "hipStreamCreate");
  halo_ok(halo_plan_upload(plan, d_meta, meta_bytes, stream), "halo_plan_upload");
  halo_ok(halo_prefix_attn_decode(plan, d_meta, d_q, d_k, d_v, d_o, d_lse, d_ws, ws_bytes, stream),
          "halo_prefix_attn_decode");
  hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");

  std::vector<unsigned char> o(rows * p.head_dim * out_elt);
  std::vector<float> lse(rows);
  hip_ok(hipMemcpy(o.data(), d_o, o.size(), hipMemcpyDeviceToHost), "copy o");
  hip_ok(hipMemcpy(lse.data(), d_lse, lse.size() * sizeof(float), hipMemcpyDeviceToHost), "copy lse");
  FILE* g = std::fopen(argv[2], "wb");
  if (!g) die("cannot open output");
  std::fwrite(o.data(), 1, o.size(), g);
  std::fwrite(lse.data(), sizeof(float), lse.size(), g);
  std::fclose(g);

  halo_plan_destroy(plan);
  for (void* d : {d_meta, d_ws, d_o, static_cast<void*>(d_lse), d_q, d_k, d_v})
    if (d) hip_ok(hipFree(d), "hipFree");
  hip_ok(hipStreamDestroy(stream), "hipStreamDestroy");
  std::printf("ok %d requests\n", R);
  return 0;
}
