// A C-ABI client of libcast.so with no Python and no torch: one block step
// (cast_route_kv -> cast_anchor_attn -> cast_par_reconstruct in accumulate mode)
// on inputs read from raw files, outputs written back as raw files.
//
//   cast_client DIR
//
// DIR/meta.txt   n_a S H dh M Bv topk scale n_frames Hg Wg D n_anchor a_0 .. a_{n_anchor-1}
// DIR/q.bin      bf16 [n_a, S, H, dh]      DIR/k.bin, DIR/v.bin  bf16 [M, Bv, H, dh]
// DIR/resid.bin  fp32 [n_frames, Hg, Wg, D]  DIR/x.bin  fp32 [n_frames, Hg, Wg, D]
// writes DIR/idx.bin (int32 [n_a, H, k_eff]), DIR/scores.bin (fp32 [n_a, H, M]),
// DIR/out.bin (bf16 [n_a, S, H, dh]), DIR/x_out.bin (fp32, X after the update).
// Exit status 0 on success; a refused call prints its status and detail.
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "../../include/cast.h"

namespace {

bool read_file(const std::string& path, std::vector<char>& buf, size_t bytes) {
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return false;
  buf.resize(bytes);
  const size_t got = bytes ? std::fread(buf.data(), 1, bytes, f) : 0;
  std::fclose(f);
  return got == bytes;
}

bool write_file(const std::string& path, const void* data, size_t bytes) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const size_t put = bytes ? std::fwrite(data, 1, bytes, f) : 0;
  std::fclose(f);
  return put == bytes;
}

// device buffer holding `bytes` (at least 256, so that every pointer is valid)
void* dev_alloc(size_t bytes) {
  void* p = nullptr;
  if (hipMalloc(&p, bytes < 256 ? 256 : bytes) != hipSuccess) return nullptr;
  return p;
}

bool hip_ok(hipError_t e, const char* what) {
  if (e == hipSuccess) return true;
  std::fprintf(stderr, "cast_client: %s: %s\n", what, hipGetErrorString(e));
  return false;
}

int fail(const char* what, int st) {
  std::fprintf(stderr, "cast_client: %s: %s (%s)\n", what, cast_status_string(st),
               cast_last_error_detail());
  return 1;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: cast_client DIR\n");
    return 2;
  }
  const std::string dir = argv[1];
  int n_a, S, H, dh, M, Bv, topk, n_frames, Hg, Wg, D, n_anchor;
  float scale;
  std::vector<int> anchors;
  {
    FILE* f = std::fopen((dir + "/meta.txt").c_str(), "r");
    if (!f || std::fscanf(f, "%d %d %d %d %d %d %d %f %d %d %d %d %d", &n_a, &S, &H, &dh, &M, &Bv,
                          &topk, &scale, &n_frames, &Hg, &Wg, &D, &n_anchor) != 13 ||
        n_anchor < 1 || n_anchor > 4096) {
      std::fprintf(stderr, "cast_client: bad meta.txt\n");
      if (f) std::fclose(f);
      return 2;
    }
    anchors.resize(n_anchor);
    for (int j = 0; j < n_anchor; ++j)
      if (std::fscanf(f, "%d", &anchors[j]) != 1) {
        std::fprintf(stderr, "cast_client: bad anchors\n");
        std::fclose(f);
        return 2;
      }
    std::fclose(f);
  }
  const size_t q_bytes = (size_t)n_a * S * H * dh * 2, kv_bytes = (size_t)M * Bv * H * dh * 2;
  const size_t fr_bytes = (size_t)n_frames * Hg * Wg * D * 4;
  std::vector<char> hq, hk, hv, hr, hx;
  if (!read_file(dir + "/q.bin", hq, q_bytes) || !read_file(dir + "/k.bin", hk, kv_bytes) ||
      !read_file(dir + "/v.bin", hv, kv_bytes) || !read_file(dir + "/resid.bin", hr, fr_bytes) ||
      !read_file(dir + "/x.bin", hx, fr_bytes)) {
    std::fprintf(stderr, "cast_client: missing or short input files\n");
    return 2;
  }
  const int k_cap = topk < M ? topk : M;
  void* q = dev_alloc(q_bytes);
  void* k = dev_alloc(kv_bytes);
  void* v = dev_alloc(kv_bytes);
  void* out = dev_alloc(q_bytes);
  float* resid = static_cast<float*>(dev_alloc(fr_bytes));
  float* x = static_cast<float*>(dev_alloc(fr_bytes));
  float* scores = static_cast<float*>(dev_alloc((size_t)n_a * H * M * 4));
  int32_t* idx = static_cast<int32_t*>(dev_alloc((size_t)n_a * H * (k_cap > 0 ? k_cap : 1) * 4));
  if (!q || !k || !v || !out || !resid || !x || !scores || !idx) {
    std::fprintf(stderr, "cast_client: hipMalloc failed\n");
    return 1;
  }
  if (!hip_ok(hipMemcpy(q, hq.data(), q_bytes, hipMemcpyHostToDevice), "copy q") ||
      !hip_ok(hipMemcpy(k, hk.data(), kv_bytes, hipMemcpyHostToDevice), "copy k") ||
      !hip_ok(hipMemcpy(v, hv.data(), kv_bytes, hipMemcpyHostToDevice), "copy v") ||
      !hip_ok(hipMemcpy(resid, hr.data(), fr_bytes, hipMemcpyHostToDevice), "copy resid") ||
      !hip_ok(hipMemcpy(x, hx.data(), fr_bytes, hipMemcpyHostToDevice), "copy x"))
    return 1;
  hipStream_t stream;
  if (!hip_ok(hipStreamCreate(&stream), "hipStreamCreate")) return 1;

  // routing
  int k_eff = -1;
  const size_t wr = cast_route_kv_workspace_bytes(n_a, S, H, dh, M, Bv);
  void* ws_route = dev_alloc(wr);
  int st = cast_route_kv(q, k, n_a, S, H, dh, M, Bv, topk, scale, scores, idx, &k_eff, ws_route, wr,
                         stream);
  if (st != CAST_OK) return fail("cast_route_kv", st);
  // attention (with the key-split workspace when the sizes use one)
  const size_t wa = cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, 0, Bv);
  void* ws_attn = wa ? dev_alloc(wa) : nullptr;
  st = cast_anchor_attn(q, k, v, idx, k_eff, nullptr, nullptr, 0, n_a, S, H, dh, M, Bv, scale, out,
                        nullptr, ws_attn, wa, stream);
  if (st != CAST_OK) return fail("cast_anchor_attn", st);
  // PAR, accumulate mode: X_t += R~_t for every skipped frame
  cast_par_params_t prm;
  cast_par_params_default(&prm);
  prm.accumulate = 1;
  const size_t wp = cast_par_workspace_bytes(n_frames, n_anchor, Hg, Wg, D, &prm);
  void* ws_par = dev_alloc(wp);
  st = cast_par_reconstruct(resid, anchors.data(), n_anchor, n_frames, Hg, Wg, D, &prm, x, nullptr,
                            nullptr, nullptr, ws_par, wp, stream);
  if (st != CAST_OK) return fail("cast_par_reconstruct", st);
  if (!hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize")) return 1;

  std::vector<char> h_idx((size_t)n_a * H * k_eff * 4), h_sc((size_t)n_a * H * M * 4);
  if (!hip_ok(hipMemcpy(h_idx.data(), idx, h_idx.size(), hipMemcpyDeviceToHost), "copy idx") ||
      !hip_ok(hipMemcpy(h_sc.data(), scores, h_sc.size(), hipMemcpyDeviceToHost), "copy scores") ||
      !hip_ok(hipMemcpy(hq.data(), out, q_bytes, hipMemcpyDeviceToHost), "copy out") ||
      !hip_ok(hipMemcpy(hx.data(), x, fr_bytes, hipMemcpyDeviceToHost), "copy x"))
    return 1;
  if (!write_file(dir + "/idx.bin", h_idx.data(), h_idx.size()) ||
      !write_file(dir + "/scores.bin", h_sc.data(), h_sc.size()) ||
      !write_file(dir + "/out.bin", hq.data(), q_bytes) ||
      !write_file(dir + "/x_out.bin", hx.data(), fr_bytes)) {
    std::fprintf(stderr, "cast_client: cannot write outputs\n");
    return 1;
  }
  for (void* p : {q, k, v, out, (void*)resid, (void*)x, (void*)scores, (void*)idx, ws_route,
                  ws_attn, ws_par})
    if (p && !hip_ok(hipFree(p), "hipFree")) return 1;
  if (!hip_ok(hipStreamDestroy(stream), "hipStreamDestroy")) return 1;
  std::printf("cast_client ok: k_eff %d, ABI %d\n", k_eff, cast_abi_version());
  return 0;
}
