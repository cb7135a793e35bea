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
//
// With a third argument STEPS, a decode loop: the plan is made for the batch
// with every private segment (on one path, longer than STEPS) STEPS tokens
// shorter, then each step appends a token to each of them (the pages they
// reopen come back from the input's page lists), brings the plan up to date
// (halo_plan_update_lengths + halo_plan_upload_update, or a new plan), and
// decodes. The output is the last step's, i.e. the input batch's. Prints the
// steps updated in place and the median host time per step (update, upload
// and decode launches).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <chrono>
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
  if (argc != 3 && argc != 4) die("usage: decode INPUT OUTPUT [STEPS]");
  const int steps = argc == 4 ? std::atoi(argv[3]) : 0;
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

  // The loop's forests: lengths `len`, each segment's first ceil(len / 16)
  // input pages.
  std::vector<int32_t> refs(S, 0);
  for (int32_t s : req_seg_ids) refs[s]++;
  std::vector<int32_t> cur_len = seg_len, cur_indptr(S + 1, 0), cur_ids;
  for (int s = 0; s < S; ++s)
    if (steps > 0 && refs[s] == 1 && seg_len[s] > steps) cur_len[s] -= steps;
  halo_forest_t forest{};
  auto make_forest = [&]() {
    cur_ids.clear();
    for (int s = 0; s < S; ++s) {
      const int32_t np = (cur_len[s] + 15) / 16;
      cur_ids.insert(cur_ids.end(), seg_page_ids.begin() + seg_page_indptr[s],
                     seg_page_ids.begin() + seg_page_indptr[s] + np);
      cur_indptr[s + 1] = cur_indptr[s] + np;
    }
    forest.num_segments = S;
    forest.seg_len = cur_len.data();
    forest.seg_page_indptr = cur_indptr.data();
    forest.seg_page_ids = cur_ids.data();
    forest.num_requests = R;
    forest.req_seg_indptr = req_seg_indptr.data();
    forest.req_seg_ids = req_seg_ids.data();
    forest.q_len = nullptr;
  };
  make_forest();

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
  int in_place = 0;
  std::vector<double> host_us;
  if (steps > 0) {
    // Double-buffered metadata: step t + 1's upload goes into the buffer the
    // running step does not read, on a copy stream, after the last decode
    // that read that buffer; a decode waits for its buffer's upload.
    void* metas[2] = {d_meta, nullptr};
    size_t meta_cap[2] = {meta_bytes, 0};
    const halo_plan_t* holds[2] = {plan, nullptr};   // the plan whose upload buffer i holds
    hipStream_t copy;
    hip_ok(hipStreamCreate(&copy), "hipStreamCreate");
    hipEvent_t uploaded[2], ran[2];
    for (int i = 0; i < 2; ++i) {
      hip_ok(hipEventCreateWithFlags(&uploaded[i], hipEventDisableTiming), "hipEventCreate");
      hip_ok(hipEventCreateWithFlags(&ran[i], hipEventDisableTiming), "hipEventCreate");
    }
    hip_ok(hipEventRecord(uploaded[0], stream), "hipEventRecord");
    hip_ok(hipEventRecord(ran[0], stream), "hipEventRecord");
    hip_ok(hipEventRecord(ran[1], stream), "hipEventRecord");
    int cur = 0;
    for (int t = 0; t < steps; ++t) {
      for (int s = 0; s < S; ++s)
        if (cur_len[s] < seg_len[s]) cur_len[s]++;
      make_forest();
      const auto t0 = std::chrono::steady_clock::now();
      // the last upload read the host image
      hip_ok(hipEventSynchronize(uploaded[cur]), "hipEventSynchronize");
      const halo_status_t st = halo_plan_update_lengths(plan, &forest);
      if (st == HALO_OK) {
        ++in_place;
      } else {
        if (st != HALO_ERR_REPLAN) halo_ok(st, "halo_plan_update_lengths");
        halo_plan_destroy(plan);
        size_t wb = 0;
        halo_ok(halo_plan_create(&p, &forest, &plan, &meta_bytes, &wb), "halo_plan_create");
        if (wb > ws_bytes) {
          hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
          hip_ok(hipFree(d_ws), "hipFree");
          hip_ok(hipMalloc(&d_ws, wb), "hipMalloc workspace");
          ws_bytes = wb;
        }
        holds[0] = holds[1] = nullptr;
      }
      const int nxt = 1 - cur;
      if (meta_cap[nxt] < meta_bytes) {
        hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize");
        if (metas[nxt]) hip_ok(hipFree(metas[nxt]), "hipFree");
        hip_ok(hipMalloc(&metas[nxt], meta_bytes), "hipMalloc meta");
        meta_cap[nxt] = meta_bytes;
        holds[nxt] = nullptr;
      }
      hip_ok(hipStreamWaitEvent(copy, ran[nxt], 0), "hipStreamWaitEvent");
      if (holds[nxt] == plan) {
        halo_ok(halo_plan_upload_update(plan, metas[nxt], meta_cap[nxt], copy), "halo_plan_upload_update");
      } else {
        halo_ok(halo_plan_upload(plan, metas[nxt], meta_cap[nxt], copy), "halo_plan_upload");
        holds[nxt] = plan;
      }
      hip_ok(hipEventRecord(uploaded[nxt], copy), "hipEventRecord");
      hip_ok(hipStreamWaitEvent(stream, uploaded[nxt], 0), "hipStreamWaitEvent");
      halo_ok(halo_prefix_attn_decode(plan, metas[nxt], d_q, d_k, d_v, d_o, d_lse, d_ws, ws_bytes, stream),
              "halo_prefix_attn_decode");
      hip_ok(hipEventRecord(ran[nxt], stream), "hipEventRecord");
      cur = nxt;
      host_us.push_back(std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count());
    }
    hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");
    hip_ok(hipStreamSynchronize(copy), "hipStreamSynchronize");
    for (int i = 0; i < 2; ++i) {
      hip_ok(hipEventDestroy(uploaded[i]), "hipEventDestroy");
      hip_ok(hipEventDestroy(ran[i]), "hipEventDestroy");
    }
    hip_ok(hipStreamDestroy(copy), "hipStreamDestroy");
    d_meta = metas[0];
    if (metas[1]) hip_ok(hipFree(metas[1]), "hipFree");
  }
  hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize");
  if (steps > 0) {
    std::sort(host_us.begin(), host_us.end());
    std::printf("loop steps %d in_place %d host_us_median %.1f\n", steps, in_place, host_us[host_us.size() / 2]);
  }

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
