// Host-side driver for the AddressSanitizer / UndefinedBehaviorSanitizer build
// of librp's host code (the C-ABI validation in rp_api.hip and the scheduling
// simulation in rp_sched.cpp). Built and run by tests/test_sanitize_host.py.
//
// Every call either fails validation before reaching the HIP runtime (fake,
// aligned device addresses that are never dereferenced), runs host code only
// (rp_sched_simulate, rp_plan_layout), or, only when the runtime reports no
// GPU, reaches the runtime and must come back as RP_ERR_HIP. Exit status 0
// means every expectation held and the sanitizers reported nothing.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "rp.h"

namespace {

int g_fail = 0;
#define EXPECT(cond)                                                             \
  do {                                                                           \
    if (!(cond)) {                                                               \
      std::fprintf(stderr, "FAILED %s:%d: %s (last error: %s)\n", __FILE__,     \
                   __LINE__, #cond, rp_last_error());                            \
      ++g_fail;                                                                  \
    }                                                                            \
  } while (0)

void* const A = reinterpret_cast<void*>(uintptr_t(0x10000000));
void* at(size_t off) { return static_cast<char*>(A) + off; }

rp_paged_kv kv_ok() {
  rp_paged_kv kv{};
  kv.k_pages = A;
  kv.v_pages = at(4096);
  kv.num_pages = 4;
  kv.num_kv_heads = 2;
  kv.page_size = 16;
  kv.head_dim = 64;
  kv.kv_dtype = RP_KV_BF16;
  return kv;
}

rp_group_layout layout_ok(int S = 2, int G = 1, int mpp = 2, int mrp = 2) {
  rp_group_layout l{};
  l.num_seqs = S;
  l.num_groups = G;
  l.num_q_heads = 4;
  l.seq_to_group = static_cast<const int32_t*>(A);
  l.prefix_lens = static_cast<const int32_t*>(A);
  l.prefix_block_table = static_cast<const int32_t*>(A);
  l.max_prefix_pages = mpp;
  l.resp_lens = static_cast<const int32_t*>(A);
  l.resp_block_table = static_cast<const int32_t*>(A);
  l.max_resp_pages = mrp;
  return l;
}

void status_strings() {
  for (int s = 0; s <= 6; ++s) EXPECT(rp_status_string(static_cast<rp_status>(s)) != nullptr);
  EXPECT(std::strstr(rp_status_string(static_cast<rp_status>(99)), "unknown") != nullptr);
  EXPECT(rp_last_error() != nullptr);
}

void validation() {
  rp_paged_kv kv = kv_ok();
  rp_group_layout l = layout_ok();
  size_t n = 0;
  EXPECT(rp_group_decode_attn_workspace_size(nullptr, &l, &n) == RP_ERR_INVALID_ARG);
  EXPECT(rp_group_decode_attn_workspace_size(&kv, nullptr, &n) == RP_ERR_INVALID_ARG);
  EXPECT(rp_group_decode_attn_workspace_size(&kv, &l, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_group_decode_attn_workspace_size(&kv, &l, &n) == RP_OK && n > 0);
  const size_t need = n;

  // Every field of the pool and the layout, one bad value at a time.
  struct KvCase { void (*mut)(rp_paged_kv&); rp_status want; };
  const KvCase kv_cases[] = {
      {[](rp_paged_kv& k) { k.k_pages = nullptr; }, RP_ERR_INVALID_ARG},
      {[](rp_paged_kv& k) { k.v_pages = at(8); }, RP_ERR_INVALID_ARG},
      {[](rp_paged_kv& k) { k.page_size = 32; }, RP_ERR_UNSUPPORTED},
      {[](rp_paged_kv& k) { k.head_dim = 96; }, RP_ERR_UNSUPPORTED},
      {[](rp_paged_kv& k) { k.kv_dtype = RP_KV_FP8_E4M3; }, RP_ERR_INVALID_ARG},
      {[](rp_paged_kv& k) { k.k_scale = static_cast<float*>(A); }, RP_ERR_INVALID_ARG},
      {[](rp_paged_kv& k) { k.kv_dtype = static_cast<rp_kv_dtype>(7); }, RP_ERR_UNSUPPORTED},
      {[](rp_paged_kv& k) { k.num_pages = 0; }, RP_ERR_INVALID_ARG},
      {[](rp_paged_kv& k) { k.num_kv_heads = 0; }, RP_ERR_INVALID_ARG},
  };
  for (const KvCase& c : kv_cases) {
    rp_paged_kv k = kv_ok();
    c.mut(k);
    EXPECT(rp_group_decode_attn_workspace_size(&k, &l, &n) == c.want);
    EXPECT(rp_plan(&k, &l, A, need, nullptr) == c.want);
    EXPECT(rp_kv_append(&k, &l, A, A, nullptr) == c.want);
  }
  struct LayCase { void (*mut)(rp_group_layout&); rp_status want; };
  const LayCase lay_cases[] = {
      {[](rp_group_layout& x) { x.num_q_heads = 3; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.num_q_heads = 6; }, RP_ERR_UNSUPPORTED},
      {[](rp_group_layout& x) { x.num_q_heads = 0; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.num_groups = 0; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.num_groups = 4097; }, RP_ERR_UNSUPPORTED},
      {[](rp_group_layout& x) { x.seq_to_group = nullptr; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.resp_block_table = nullptr; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.num_seqs = -1; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.max_resp_pages = -1; }, RP_ERR_INVALID_ARG},
      {[](rp_group_layout& x) { x.num_seqs = 1 << 20; x.max_resp_pages = 1 << 12; }, RP_ERR_UNSUPPORTED},
  };
  for (const LayCase& c : lay_cases) {
    rp_group_layout x = layout_ok();
    c.mut(x);
    EXPECT(rp_group_decode_attn_workspace_size(&kv, &x, &n) == c.want);
    EXPECT(rp_group_decode_attn(&kv, &x, A, 0.1f, A, nullptr, A, need, nullptr) == c.want);
  }

  // Workspace and pointer checks.
  EXPECT(rp_plan(&kv, &l, A, need - 1, nullptr) == RP_ERR_WORKSPACE);
  EXPECT(rp_plan(&kv, &l, at(64), need, nullptr) == RP_ERR_WORKSPACE);
  EXPECT(rp_plan(&kv, &l, nullptr, need, nullptr) == RP_ERR_WORKSPACE);
  EXPECT(rp_group_decode_attn(&kv, &l, nullptr, 0.1f, A, nullptr, A, need, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_group_decode_attn(&kv, &l, A, 0.1f, at(2), nullptr, A, need, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_group_decode_attn(&kv, &l, A, 0.1f, A, static_cast<float*>(at(2)), A, need, nullptr) ==
         RP_ERR_INVALID_ARG);
  EXPECT(rp_attn_parts(&kv, &l, at(4), 0.1f, A, need, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_combine_parts(&kv, &l, nullptr, nullptr, A, need, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_kv_append(&kv, &l, nullptr, A, nullptr) == RP_ERR_INVALID_ARG);
  rp_group_layout no_resp = layout_ok(2, 1, 2, 0);
  EXPECT(rp_kv_append(&kv, &no_resp, A, A, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_lse_combine(static_cast<const float*>(A), static_cast<const float*>(A),
                        static_cast<const int32_t*>(A), 4, 96, A, nullptr, nullptr) == RP_ERR_UNSUPPORTED);
  EXPECT(rp_lse_combine(static_cast<const float*>(A), static_cast<const float*>(A), nullptr, 4, 128, A,
                        nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_lse_combine(nullptr, nullptr, nullptr, -1, 128, nullptr, nullptr, nullptr) == RP_ERR_INVALID_ARG);

  // Empty batches return before touching any pointer.
  rp_group_layout empty = layout_ok(0);
  EXPECT(rp_group_decode_attn_workspace_size(&kv, &empty, &n) == RP_OK && n == 0);
  EXPECT(rp_group_decode_attn(&kv, &empty, nullptr, 0.1f, nullptr, nullptr, nullptr, 0, nullptr) == RP_OK);
  EXPECT(rp_kv_append(&kv, &empty, nullptr, nullptr, nullptr) == RP_OK);
  EXPECT(rp_lse_combine(nullptr, nullptr, nullptr, 0, 128, nullptr, nullptr, nullptr) == RP_OK);

  // q/k prep, GRPO and prefill argument checks.
  EXPECT(rp_decode_qk_prep(&kv, &l, nullptr, A, A, A, A, 1e-6, 1e6, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_decode_qk_prep(&kv, &l, A, A, A, A, A, -1.0, 1e6, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_decode_qk_prep(&kv, &l, A, A, A, A, A, NAN, 1e6, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_decode_qk_prep(&kv, &l, A, A, A, A, A, 1e-6, 0.0, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_decode_qk_prep(&kv, &l, A, A, A, A, A, 1e-6, 1e6, A, at(1), nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_grpo_advantage(nullptr, 4, 8, 1e-6, 1, static_cast<float*>(A), nullptr, nullptr, nullptr) ==
         RP_ERR_INVALID_ARG);
  EXPECT(rp_grpo_advantage(static_cast<const float*>(A), 4, 8, 1e-6, 2, static_cast<float*>(A), nullptr, nullptr,
                           nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_grpo_advantage(static_cast<const float*>(A), 4, 0, 1e-6, 1, static_cast<float*>(A), nullptr, nullptr,
                           nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_grpo_advantage(nullptr, 0, 8, 1e-6, 1, nullptr, nullptr, nullptr, nullptr) == RP_OK);
  EXPECT(rp_selftest_mfma(9, A, A, static_cast<float*>(A), nullptr) == RP_ERR_UNSUPPORTED);
  EXPECT(rp_selftest_mfma(0, nullptr, A, static_cast<float*>(A), nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_stream_read(A, 24, static_cast<uint32_t*>(A), 0, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_stream_read(nullptr, 1024, static_cast<uint32_t*>(A), 1, nullptr) == RP_ERR_INVALID_ARG);
  rp_prefill_layout pl{2, 4, 10, static_cast<const int32_t*>(A), static_cast<const int32_t*>(A), 2};
  EXPECT(rp_prefill_kv_write(&kv, &pl, nullptr, A, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_prefill_attn(&kv, &pl, A, A, A, 0.0f, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_prefill(&kv, &pl, A, A, A, INFINITY, A, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  EXPECT(rp_prefill(&kv, &pl, A, A, A, 0.1f, nullptr, nullptr, nullptr) == RP_ERR_INVALID_ARG);
  rp_prefill_layout bad = pl;
  bad.prompt_offs = nullptr;
  EXPECT(rp_prefill_kv_write(&kv, &bad, A, A, nullptr) == RP_ERR_INVALID_ARG);
  bad = pl;
  bad.num_q_heads = 6;
  EXPECT(rp_prefill_attn(&kv, &bad, A, A, A, 0.1f, A, nullptr, nullptr) == RP_ERR_UNSUPPORTED);

  // Plan layouts (host arithmetic only) over a sweep of shapes: sections ordered, aligned, inside
  // the workspace.
  for (int S : {1, 7, 256, 1024, 8500})
    for (int mrp : {0, 1, 70, 1025, 2049})
      for (int D : {64, 128}) {
        rp_paged_kv k = kv_ok();
        k.head_dim = D;
        k.num_kv_heads = 8;
        rp_group_layout x = layout_ok(S, S < 64 ? S : 64, 64, mrp);
        x.num_q_heads = 16;
        rp_plan_info info{};
        size_t ws = 0;
        EXPECT(rp_plan_layout(&k, &x, &info) == RP_OK);
        EXPECT(rp_group_decode_attn_workspace_size(&k, &x, &ws) == RP_OK);
        const size_t offs[] = {info.hdr, info.grp_off, info.grp_members, info.prefix_items,
                               info.resp_items, info.seq_parts, info.part_o, info.part_lse};
        for (size_t i = 0; i < 8; ++i) {
          EXPECT(offs[i] % 256 == 0);
          if (i) EXPECT(offs[i] >= offs[i - 1]);  // an empty section takes no bytes
        }
        EXPECT(info.part_lse + 4 * (size_t)info.max_parts <= ws);
      }
}

void sched() {
  std::mt19937 gen(7);
  for (int mode = 0; mode < 3; ++mode)
    for (int R : {1, 4, 12, 96})
      for (int K : {1, 8})
        for (int U : {1, 2}) {
          if (R % U) continue;
          std::vector<int32_t> P(R), L(R * K);
          for (auto& p : P) p = (int32_t)(gen() % 1024);
          for (auto& x : L) x = 1 + (int32_t)(gen() % 5000);
          rp_sched_config c{};
          c.mode = static_cast<rp_sched_mode>(mode);
          c.num_groups = R;
          c.group_size = K;
          c.update_groups = U;
          c.frontier_width = 2;
          c.max_running = 1 + (int32_t)(gen() % 300);
          c.step_base = 1e-3;
          c.step_per_seq = 2.7e-6;
          c.step_per_ctx_token = 1.7e-8;
          c.prefill_per_token = 2e-7;
          c.mat_base = 1.0;
          c.train_per_token = 1e-4;
          c.opt_step = 0.5;
          rp_sched_summary s{};
          std::vector<double> done(R), enter(R), trainable(R), ustart(R / U), uend(R / U);
          std::vector<int32_t> fifo(R);
          EXPECT(rp_sched_simulate(&c, P.data(), L.data(), &s, done.data(), enter.data(), trainable.data(),
                                   fifo.data(), ustart.data(), uend.data()) == RP_OK);
          EXPECT(s.t_train_end >= s.t_complete && s.steps > 0 && std::isfinite(s.wait_ratio));
          // Outputs optional.
          rp_sched_summary s2{};
          EXPECT(rp_sched_simulate(&c, P.data(), L.data(), &s2, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr) == RP_OK);
          EXPECT(s2.t_train_end == s.t_train_end);
        }
  // Invalid configurations are refused.
  std::vector<int32_t> P(4, 10), L(8, 5);
  rp_sched_config c{};
  c.mode = RP_SCHED_CGP;
  c.num_groups = 4;
  c.group_size = 2;
  c.update_groups = 3;
  c.max_running = 4;
  rp_sched_summary s{};
  EXPECT(rp_sched_simulate(&c, P.data(), L.data(), &s, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) !=
         RP_OK);
  c.update_groups = 2;
  c.step_base = -1.0;
  EXPECT(rp_sched_simulate(&c, P.data(), L.data(), &s, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) !=
         RP_OK);
  c.step_base = 0.0;
  L[3] = 0;
  EXPECT(rp_sched_simulate(&c, P.data(), L.data(), &s, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) !=
         RP_OK);
  EXPECT(rp_sched_simulate(nullptr, P.data(), L.data(), &s, nullptr, nullptr, nullptr, nullptr, nullptr,
                           nullptr) != RP_OK);
}

// Only on a host without a GPU: a well-formed call reaches the runtime, which fails.
void runtime_failure() {
  int n = -1;
  const hipError_t e = hipGetDeviceCount(&n);
  if (e == hipSuccess && n > 0) {
    std::printf("runtime_failure: skipped (%d GPU(s) visible)\n", n);
    return;
  }
  rp_paged_kv kv = kv_ok();
  rp_group_layout l = layout_ok();
  size_t need = 0;
  EXPECT(rp_group_decode_attn_workspace_size(&kv, &l, &need) == RP_OK);
  EXPECT(rp_plan(&kv, &l, A, need, nullptr) == RP_ERR_HIP);
  EXPECT(std::strstr(rp_last_error(), "hipGetDevice") != nullptr);
  EXPECT(rp_kv_append(&kv, &l, A, A, nullptr) == RP_ERR_HIP);
  EXPECT(rp_lse_combine(static_cast<const float*>(A), static_cast<const float*>(A),
                        static_cast<const int32_t*>(A), 4, 64, A, nullptr, nullptr) == RP_ERR_HIP);
  EXPECT(rp_validate_layout(&kv, &l, nullptr) == RP_ERR_HIP);
}

}  // namespace

int main() {
  status_strings();
  validation();
  sched();
  runtime_failure();
  if (g_fail) {
    std::fprintf(stderr, "%d expectation(s) failed\n", g_fail);
    return 1;
  }
  std::printf("sanitize_host: all expectations held\n");
  return 0;
}
