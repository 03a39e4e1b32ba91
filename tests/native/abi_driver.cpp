// Host-side exercise of the C ABI for sanitizer builds (AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code of libcommitkv_asan.so and of
// this program; device code is built as usual).  Every entry point runs on
// small seeded inputs, including its argument-error paths, and an agent runs
// a short episode through commits, posts and checkpoints.  Results are not
// compared with anything here (the parity tests do that): the program checks
// return codes and leaves memory errors to the sanitizers.
//
// Exit status 0 when every call returned what it should.
#include "commitkv.h"
#include "commitkv_agent.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

namespace {

int g_fail = 0;

void expect(int rc, int want, const char* what, ckv_ctx* c) {
  if (rc != want) {
    std::fprintf(stderr, "[driver] %s: returned %d, expected %d (%s)\n", what, rc, want,
                 c ? ckv_last_error(c) : "");
    ++g_fail;
  }
}

template <class T>
T* dev_copy(const std::vector<T>& h) {
  T* d = nullptr;
  if (hipMalloc(&d, std::max<size_t>(h.size(), 1) * sizeof(T)) != hipSuccess) return nullptr;
  if (!h.empty()) (void)hipMemcpy(d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice);
  return d;
}

template <class T>
T* dev_zeros(size_t n) {
  T* d = nullptr;
  if (hipMalloc(&d, std::max<size_t>(n, 1) * sizeof(T)) != hipSuccess) return nullptr;
  (void)hipMemset(d, 0, std::max<size_t>(n, 1) * sizeof(T));
  return d;
}

// bf16 bits of normal(0, sd) draws
std::vector<uint16_t> bf16_normal(size_t n, double sd, std::mt19937_64& rng) {
  std::normal_distribution<float> nd(0.f, (float)sd);
  std::vector<uint16_t> out(n);
  for (size_t i = 0; i < n; ++i) {
    const float f = nd(rng);
    uint32_t b;
    std::memcpy(&b, &f, 4);
    out[i] = (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
  }
  return out;
}

}  // namespace

int main() {
  std::mt19937_64 rng(20261202);
  ckv_ctx* c = nullptr;
  expect(ckv_create(&c, 0, nullptr), CKV_OK, "ckv_create", nullptr);
  if (!c) return 1;
  std::printf("[driver] version %u, build flags %u\n", ckv_version(), ckv_build_flags());

  // one layer: 2 KV heads, 8 query heads, d = 64, S = 1536 tokens, W = 16
  const int Hkv = 2, Hq = 8, D = 64, S = 1536, W = 16, G = 16;
  std::vector<uint16_t> hk = bf16_normal((size_t)Hkv * S * D, 1.0, rng);
  std::vector<uint16_t> hv = bf16_normal((size_t)Hkv * S * D, 1.0, rng);
  std::vector<uint16_t> hq = bf16_normal((size_t)Hq * W * D, 1.0, rng);
  std::vector<int32_t> hpos(S), hqpos(W);
  for (int t = 0; t < S; ++t) hpos[t] = t;
  for (int p = 0; p < W; ++p) hqpos[p] = S - W + p;
  uint16_t* k = dev_copy(hk);
  uint16_t* v = dev_copy(hv);
  uint16_t* q = dev_copy(hq);
  int32_t* pos = dev_copy(hpos);
  int32_t* qpos = dev_copy(hqpos);
  const ckv_kv_view kv{k, v, (int64_t)S * D, D, pos, S, Hkv, D, nullptr, 0};
  const ckv_window_view win{q, (int64_t)W * D, D, qpos, Hq, W, 0.f};
  // pages of G tokens over the first S - 2W tokens, some shorter
  std::vector<int32_t> st, ln;
  for (int t = 0; t + G <= S - 2 * W; t += G) {
    st.push_back(t);
    ln.push_back((t / G) % 5 == 3 ? G / 2 : G);
  }
  const int n = (int)st.size();
  const ckv_page_list pages{st.data(), ln.data(), n};
  float* R = dev_zeros<float>(n);
  float* R2 = dev_zeros<float>(n);
  float* Rh = dev_zeros<float>((size_t)n * Hq);
  float* o = dev_zeros<float>((size_t)Hq * W * D);
  float* lse = dev_zeros<float>((size_t)Hq * W);
  float* mass = dev_zeros<float>(S);

  // measurement: every output, then the allocation-free form, then a batch
  expect(ckv_measure_page_effects(c, &kv, &win, &pages, R, Rh, o, lse, mass), CKV_OK, "measure", c);
  expect(ckv_measure_page_effects_noalloc(c, &kv, &win, &pages, R2, nullptr, nullptr, nullptr, nullptr), CKV_OK,
         "measure_noalloc", c);
  {
    const ckv_kv_view kvs[2] = {kv, kv};
    const ckv_window_view wins[2] = {win, win};
    const ckv_page_list pls[2] = {pages, pages};
    float* Rs[2] = {R, R2};
    expect(ckv_measure_page_effects_batch(c, 2, kvs, wins, pls, Rs, nullptr, nullptr, nullptr, nullptr), CKV_OK,
           "measure_batch", c);
  }
  expect(ckv_measure_recorded(c, &kv, &win, &pages, o, lse, R2, nullptr, mass), CKV_OK, "measure_recorded", c);
  // argument errors
  expect(ckv_measure_page_effects(c, nullptr, &win, &pages, R, nullptr, nullptr, nullptr, nullptr), CKV_ERR_ARG,
         "measure NULL kv", c);
  {
    std::vector<int32_t> bad_st = {0, 8}, bad_ln = {16, 16};   // overlapping
    const ckv_page_list bad{bad_st.data(), bad_ln.data(), 2};
    expect(ckv_measure_page_effects(c, &kv, &win, &bad, R, nullptr, nullptr, nullptr, nullptr), CKV_ERR_SHAPE,
           "measure overlapping pages", c);
  }
  expect(ckv_sync(c), CKV_OK, "sync after measurement", c);

  // classification and the joint test
  uint8_t* lambda = dev_zeros<uint8_t>(n);
  int32_t* cand = dev_zeros<int32_t>(n);
  int32_t* ncand = dev_zeros<int32_t>(1);
  std::vector<uint8_t> hforce(n, 0);
  for (int i = 0; i < n; i += 7) hforce[i] = 1;
  uint8_t* force = dev_copy(hforce);
  expect(ckv_classify_pages(c, n, R, R2, nullptr, force, n, lambda, nullptr, nullptr, cand, ncand), CKV_OK,
         "classify", c);
  uint8_t* acc = dev_zeros<uint8_t>(n);
  float* uR = dev_zeros<float>(n);
  int32_t* nacc = dev_zeros<int32_t>(1);
  expect(ckv_joint_test(c, &kv, &win, o, lse, &pages, cand, ncand, n, 0.01f, acc, uR, nacc), CKV_OK, "joint", c);
  expect(ckv_joint_test(c, &kv, &win, o, lse, &pages, cand, ncand, 0, 0.01f, acc, uR, nacc), CKV_ERR_SHAPE,
         "joint max_cand 0", c);

  // pooled score, then selection and compaction of two sequences
  float* pooled = dev_zeros<float>(S);
  const int32_t nt_h = S;
  int32_t* nt = dev_copy(std::vector<int32_t>{nt_h});
  expect(ckv_pool_scores(c, mass, pooled, 1, S, nt, 7, CKV_POOL_MAX), CKV_OK, "pool", c);
  {
    const int L = 2, cap = S, B = 512;
    std::vector<uint16_t> hc = bf16_normal((size_t)2 * L * Hkv * cap * D, 1.0, rng);
    uint16_t* ck = dev_copy(hc);
    uint16_t* cv = dev_copy(hc);
    std::vector<int32_t> hp(2 * cap);
    for (int i = 0; i < 2 * cap; ++i) hp[i] = i % cap;
    int32_t* cpos = dev_copy(hp);
    const int64_t tok = D, head = (int64_t)cap * D, layer = Hkv * head, seq = L * layer;
    ckv_cache_view in{ck, cv, seq, layer, head, tok, cpos, cap, 2, L, Hkv, D, cap};
    uint16_t* ok_ = dev_zeros<uint16_t>((size_t)2 * L * Hkv * B * D);
    uint16_t* ov_ = dev_zeros<uint16_t>((size_t)2 * L * Hkv * B * D);
    int32_t* opos = dev_zeros<int32_t>((size_t)2 * B);
    const int64_t ohead = (int64_t)B * D, olayer = Hkv * ohead, oseq = L * olayer;
    ckv_cache_view out{ok_, ov_, oseq, olayer, ohead, tok, opos, B, 2, L, Hkv, D, B};
    int32_t* ntok = dev_copy(std::vector<int32_t>{S, S - 100});
    std::vector<float> hs(2 * (size_t)cap);
    std::uniform_real_distribution<float> ud(0.f, 1.f);
    for (auto& x : hs) x = ud(rng);
    float* score = dev_copy(hs);
    std::vector<int32_t> rs = {32, 64}, rl = {16, 16}, ps = {128}, pl = {16};
    const ckv_page_list ret[2] = {{rs.data(), rl.data(), 2}, {nullptr, nullptr, 0}};
    const ckv_page_list pend[2] = {{ps.data(), pl.data(), 1}, {nullptr, nullptr, 0}};
    float* rpre = dev_copy(std::vector<float>{0.5f});
    const float* rp[2] = {rpre, nullptr};
    const ckv_budget bg{B, 0.125f, 16, 8};
    int32_t* kept = dev_zeros<int32_t>((size_t)2 * B);
    int32_t* nkept = dev_zeros<int32_t>(2);
    uint8_t* state = dev_zeros<uint8_t>((size_t)2 * cap);
    expect(ckv_select_and_compact(c, &in, ntok, score, cap, ret, pend, rp, nullptr, &bg, &out, kept, nkept, state),
           CKV_OK, "select_and_compact", c);
    const ckv_budget big{B + 1, 0.125f, 16, 8};
    expect(ckv_select_and_compact(c, &in, ntok, score, cap, ret, pend, rp, nullptr, &big, &out, kept, nkept, state),
           CKV_ERR_SHAPE, "select_and_compact capacity < B", c);
    expect(ckv_sync(c), CKV_OK, "sync after selection", c);
    for (void* p : {(void*)ck, (void*)cv, (void*)cpos, (void*)ok_, (void*)ov_, (void*)opos, (void*)ntok, (void*)score,
                    (void*)rpre, (void*)kept, (void*)nkept, (void*)state})
      (void)hipFree(p);
  }

  // an agent episode: prompt, then turns of reasoning, tool call (commit),
  // observation, reasoning (post), with checkpoints when due
  {
    const int L = 2, cap = 4096, B = 1024, WA = 16, HqA = 8;
    std::vector<uint16_t> zero((size_t)L * Hkv * cap * D, 0);
    uint16_t* k0 = dev_copy(zero);
    uint16_t* v0 = dev_copy(zero);
    uint16_t* k1 = dev_copy(zero);
    uint16_t* v1 = dev_copy(zero);
    int32_t* p0 = dev_zeros<int32_t>(cap);
    int32_t* p1 = dev_zeros<int32_t>(cap);
    const int64_t head = (int64_t)cap * D, layer = Hkv * head;
    const ckv_cache_view b0{k0, v0, L * layer, layer, head, D, p0, cap, 1, L, Hkv, D, cap};
    const ckv_cache_view b1{k1, v1, L * layer, layer, head, D, p1, cap, 1, L, Hkv, D, cap};
    ckv_agent_config cfg{};
    cfg.page_size = 16;
    cfg.window = WA;
    cfg.n_q_heads = HqA;
    cfg.max_scan_pages = 64;
    cfg.checkpoint_every = 128;
    cfg.score_layer = 1;
    cfg.report_detail = 1;
    cfg.thresholds = ckv_thresholds{0.05f, 0.01f, 0.75f, 0.25f, 0.01f};
    cfg.budget = ckv_budget{B, 0.125f, 16, 16};
    cfg.pool_kernel = 0;
    cfg.pool_mode = CKV_POOL_MAX;
    ckv_agent* ag = nullptr;
    expect(ckv_agent_create(c, &b0, &b1, &cfg, &ag), CKV_OK, "agent_create", c);
    if (ag) {
      std::vector<uint16_t> qa = bf16_normal((size_t)HqA * WA * D, 1.0, rng);
      uint16_t* qd = dev_copy(qa);
      int32_t* qp = dev_zeros<int32_t>(WA);
      int32_t next = 0;
      auto write_tokens = [&](int n_tok) {
        // the engine's part: keys and values of the new tokens into the
        // current buffer at the resident slots
        int32_t nres = 0, which = 0;
        int64_t dec = 0;
        expect(ckv_agent_state(ag, &nres, &which, &dec), CKV_OK, "agent_state", c);
        const ckv_cache_view& bv = which ? b1 : b0;
        std::vector<uint16_t> kv_new = bf16_normal((size_t)n_tok * D, 1.0, rng);
        for (int l = 0; l < L; ++l)
          for (int g = 0; g < Hkv; ++g) {
            (void)hipMemcpy(bv.k + l * layer + g * head + (int64_t)nres * D, kv_new.data(), kv_new.size() * 2,
                            hipMemcpyHostToDevice);
            (void)hipMemcpy(bv.v + l * layer + g * head + (int64_t)nres * D, kv_new.data(), kv_new.size() * 2,
                            hipMemcpyHostToDevice);
          }
        std::vector<int32_t> pp(n_tok);
        for (int i = 0; i < n_tok; ++i) pp[i] = next + i;
        (void)hipMemcpy(bv.pos + nres, pp.data(), (size_t)n_tok * 4, hipMemcpyHostToDevice);
        return pp;
      };
      auto window_at = [&](int32_t p_end) {
        std::vector<int32_t> h(WA);
        for (int i = 0; i < WA; ++i) h[i] = p_end - WA + i;
        (void)hipMemcpy(qp, h.data(), (size_t)WA * 4, hipMemcpyHostToDevice);
        return ckv_window_view{qd, (int64_t)WA * D, D, qp, HqA, WA, 0.f};
      };
      auto append = [&](int kind, int n_tok, int decoded) {
        std::vector<int32_t> pp = write_tokens(n_tok);
        int32_t due = 0;
        expect(ckv_agent_append(ag, kind, pp.data(), n_tok, decoded, 1, &due), CKV_OK, "agent_append", c);
        next += n_tok;
        if (due & CKV_DUE_CHECKPOINT) {
          const ckv_window_view w = window_at(next);
          int32_t comp = 0;
          expect(ckv_agent_checkpoint(ag, &w, &comp), CKV_OK, "agent_checkpoint", c);
          ckv_agent_report rep{};
          expect(ckv_agent_last_report(ag, &rep), CKV_OK, "agent_last_report", c);
        }
        return due;
      };
      append(CKV_EVENT_PROMPT, 300, 0);
      for (int turn = 0; turn < 8; ++turn) {
        append(CKV_EVENT_REASONING, 40 + 7 * turn, 1);
        append(CKV_EVENT_TOOL_CALL, 48, 1);
        {
          const ckv_window_view w = window_at(next);
          expect(ckv_agent_commit(ag, &w), CKV_OK, "agent_commit", c);
        }
        append(CKV_EVENT_OBSERVATION, 200 + 50 * (turn % 3), 0);
        const int due = append(CKV_EVENT_REASONING, WA + 8, 1);
        if (due & CKV_DUE_POST) {
          const ckv_window_view w = window_at(next);
          expect(ckv_agent_post(ag, &w), CKV_OK, "agent_post", c);
          ckv_agent_report rep{};
          expect(ckv_agent_last_report(ag, &rep), CKV_OK, "agent_last_report", c);
        }
        std::vector<int32_t> s(256), l(256), r(4096);
        std::vector<float> val(256);
        int32_t cnt = 0;
        expect(ckv_agent_pages(ag, 0, s.data(), l.data(), val.data(), 256, &cnt), CKV_OK, "agent_pages", c);
        expect(ckv_agent_pages(ag, 1, s.data(), l.data(), val.data(), 256, &cnt), CKV_OK, "agent_pages", c);
        expect(ckv_agent_rows(ag, 2, r.data(), 4096, &cnt), CKV_OK, "agent_rows", c);
      }
      expect(ckv_agent_append(ag, 99, nullptr, 0, 0, 1, nullptr), CKV_ERR_ARG, "agent_append bad kind", c);
      expect(ckv_agent_destroy(ag), CKV_OK, "agent_destroy", c);
      (void)hipFree(qd);
      (void)hipFree(qp);
    }
    for (void* p : {(void*)k0, (void*)v0, (void*)k1, (void*)v1, (void*)p0, (void*)p1}) (void)hipFree(p);
  }

  expect(ckv_sync(c), CKV_OK, "final sync", c);
  for (void* p : {(void*)k, (void*)v, (void*)q, (void*)pos, (void*)qpos, (void*)R, (void*)R2, (void*)Rh, (void*)o,
                  (void*)lse, (void*)mass, (void*)lambda, (void*)cand, (void*)ncand, (void*)force, (void*)acc,
                  (void*)uR, (void*)nacc, (void*)pooled, (void*)nt})
    (void)hipFree(p);
  expect(ckv_destroy(c), CKV_OK, "ckv_destroy", nullptr);
  std::printf("[driver] %s (%d failed checks)\n", g_fail ? "FAILED" : "ok", g_fail);
  return g_fail ? 1 : 0;
}
