// Drives the library's host code (linked against stub_hip.cpp) through every
// batched entry point for the workloads given on stdin, so that the
// planner, layout and uploads run under the sanitizers without a GPU.
// One command per line; every command runs its entry point twice (the
// second call takes the plan cache's path) and prints "ok <line number>"
// or "FAIL ...":
//   ortho <iters> <compute> <in_dtype> <prescale> <q> <tile> <expect> <n> r c ...
//   save  <iters> <compute> <in_dtype> <prescale> <q> <tile> <expect> <n> r c ...
//   vjp   <iters> <compute> <in_dtype> <prescale> <q> <tile> <saved> <expect> <n> r c ...
//   conv  <dtype> <expect> <n> cin cout k s d g ...
//   convvjp <dtype> <expect> <n> cin cout k s d g ...
//   convsave <dtype> <expect> <n> cin cout k s d g ...
//   selftest <which>   (a planted violation of the stand-ins' checks: must abort)
// `expect` is the orth_status the call must return (for the workspace query
// and the call); data buffers are fake device allocations of the right size.
// With an argument N > 1 the driver reads all commands first and runs them
// in N threads at once (every thread all commands, on buffers of its own,
// selftests skipped), printing only failures and a summary: the library's
// shared state (plan cache, staging pool, per-thread side streams and
// errors) under concurrent callers, for ThreadSanitizer.
#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <iostream>
#include <sstream>
#include <string>
#include <thread>
#include <vector>

#include "../../include/orth.h"

extern "C" {
void* stub_dev_alloc(size_t bytes);
void stub_reset(void);
long stub_launches(void);
long stub_launches_total(void);
void stub_selftest(int which);
}

namespace {
std::atomic<int> g_fail{0};

void check(int rc, int expect, int line, const char* what) {
  if (rc != expect) {
    std::printf("FAIL line %d %s: returned %d, expected %d (%s)\n", line, what, rc, expect, orth_last_error());
    ++g_fail;
  }
}

size_t esz(int dt) { return dt == ORTH_BF16 ? 2 : 4; }

void run_ortho(std::istringstream& in, const std::string& kind, int line) {
  orth_bjorck_opts o{};
  int expect = 0, n = 0, saved = 0;
  in >> o.iters >> o.compute >> o.in_dtype >> o.prescale >> o.power_iters >> o.tile;
  if (kind == "vjp") in >> saved;
  in >> expect >> n;
  o.beta = 0.5f;
  o.out_dtype = ORTH_F32;
  o.saved = saved;
  std::vector<orth_mat> mats(n);
  std::vector<orth_vjp_mat> vm(n);
  size_t u_len = 0;
  for (int i = 0; i < n; ++i) {
    int r = 0, c = 0;
    in >> r >> c;
    const size_t elems = (size_t)r * c;
    void* w = stub_dev_alloc(elems * esz(o.in_dtype));
    void* out = stub_dev_alloc(elems * 4);
    mats[i] = orth_mat{w, out, r, c, c, c};
    vm[i] = orth_vjp_mat{w, stub_dev_alloc(elems * 4), stub_dev_alloc(elems * esz(o.in_dtype)), r, c, c, c, c};
    u_len += (size_t)(r < c ? r : c);
  }
  if (o.prescale == ORTH_PRESCALE_SPECTRAL) o.u = static_cast<float*>(stub_dev_alloc(u_len * 4));
  int32_t* status = static_cast<int32_t*>(stub_dev_alloc(4 * (size_t)(n > 0 ? n : 1)));
  for (int rep = 0; rep < 2; ++rep) {
    size_t need = 0;
    int rc;
    if (kind == "ortho")
      rc = orth_orthogonalize_workspace_size(mats.data(), n, &o, &need);
    else if (kind == "save")
      rc = orth_orthogonalize_save_workspace_size(mats.data(), n, &o, &need);
    else
      rc = orth_orthogonalize_vjp_workspace_size(vm.data(), n, &o, &need);
    check(rc, expect, line, "workspace size");
    if (rc) return;
    void* ws = need ? stub_dev_alloc(need) : nullptr;
    stub_reset();
    if (kind == "ortho")
      rc = orth_orthogonalize_batched(mats.data(), n, &o, ws, need, status, nullptr);
    else if (kind == "save")
      rc = orth_orthogonalize_save_batched(mats.data(), n, &o, ws, need, status, nullptr);
    else
      rc = orth_orthogonalize_vjp_batched(vm.data(), n, &o, ws, need, status, nullptr);
    check(rc, expect, line, kind.c_str());
    // a workspace one byte short is refused before anything is enqueued
    if (need && rep == 1) {
      const long before = stub_launches();
      int rc2;
      if (kind == "ortho")
        rc2 = orth_orthogonalize_batched(mats.data(), n, &o, ws, need - 1, status, nullptr);
      else if (kind == "save")
        rc2 = orth_orthogonalize_save_batched(mats.data(), n, &o, ws, need - 1, status, nullptr);
      else
        rc2 = orth_orthogonalize_vjp_batched(vm.data(), n, &o, ws, need - 1, status, nullptr);
      check(rc2, ORTH_EWORKSPACE, line, "short workspace");
      if (stub_launches() != before) {
        std::printf("FAIL line %d: launches after a refused call\n", line);
        ++g_fail;
      }
    }
  }
}

void run_conv(std::istringstream& in, const std::string& kind, int line) {
  int dtype = 0, expect = 0, n = 0;
  in >> dtype >> expect >> n;
  std::vector<orth_conv_desc> d(n);
  std::vector<orth_conv_vjp_desc> v(n);
  for (int i = 0; i < n; ++i) {
    orth_conv_geom g{};
    in >> g.cin >> g.cout >> g.k >> g.stride >> g.dilation >> g.groups;
    int32_t rr = 0, rc = 0, np = 0, pr = 0, pc = 0;
    if (orth_aoc_param_shapes(&g, &rr, &rc, &np, &pr, &pc) != ORTH_OK) rr = rc = np = pr = pc = 1;
    const size_t ng = g.groups > 0 ? (size_t)g.groups : 1;
    const size_t rko = ng * rr * rc * esz(dtype), proj = ng * (np ? np : 1) * pr * pc * esz(dtype);
    const size_t kern = (size_t)(g.cout > 0 ? g.cout : 1) * (g.cin > 0 && g.groups > 0 ? g.cin / g.groups + 1 : 1) *
                        (g.k > 0 ? g.k * g.k : 1) * esz(dtype);
    void* r = stub_dev_alloc(rko);
    void* p = stub_dev_alloc(proj);
    d[i] = orth_conv_desc{g, r, p, stub_dev_alloc(kern)};
    v[i] = orth_conv_vjp_desc{g, r, p, stub_dev_alloc(kern), stub_dev_alloc(rko), stub_dev_alloc(proj)};
  }
  for (int rep = 0; rep < 2; ++rep) {
    size_t need = 0;
    int rc;
    if (kind == "conv")
      rc = orth_build_conv_kernels_workspace_size(d.data(), n, dtype, &need);
    else if (kind == "convsave")
      rc = orth_build_conv_kernels_save_workspace_size(d.data(), n, dtype, &need);
    else
      rc = orth_build_conv_kernels_vjp_workspace_size(v.data(), n, dtype, &need);
    check(rc, expect, line, "workspace size");
    if (rc) return;
    void* ws = need ? stub_dev_alloc(need) : nullptr;
    stub_reset();
    if (kind == "conv")
      rc = orth_build_conv_kernels_batched(d.data(), n, dtype, ws, need, nullptr);
    else if (kind == "convsave")
      rc = orth_build_conv_kernels_save_batched(d.data(), n, dtype, ws, need, nullptr);
    else
      rc = orth_build_conv_kernels_vjp_batched(v.data(), n, dtype, ws, need, nullptr);
    check(rc, expect, line, kind.c_str());
    if (kind == "convsave" && rc == ORTH_OK) {
      // the saved product reads what the saving composition left
      stub_reset();
      check(orth_build_conv_kernels_vjp_saved_batched(v.data(), n, dtype, ws, need, nullptr), ORTH_OK, line,
            "saved composition VJP");
    }
  }
}

// one command line; returns false for a blank line or a comment
bool run_line(const std::string& text, int line, bool threaded) {
  std::istringstream in(text);
  std::string kind;
  if (!(in >> kind) || kind[0] == '#') return false;
  if (kind == "ortho" || kind == "save" || kind == "vjp")
    run_ortho(in, kind, line);
  else if (kind == "conv" || kind == "convvjp" || kind == "convsave")
    run_conv(in, kind, line);
  else if (kind == "selftest") {
    int which = 0;
    in >> which;
    if (!threaded) stub_selftest(which);
  } else {
    std::printf("FAIL line %d: unknown command %s\n", line, kind.c_str());
    ++g_fail;
  }
  return true;
}
}  // namespace

int main(int argc, char** argv) {
  const int threads = argc > 1 ? std::atoi(argv[1]) : 1;
  std::vector<std::string> lines;
  for (std::string text; std::getline(std::cin, text);) lines.push_back(text);
  if (threads > 1) {
    std::atomic<int> done{0};
    std::vector<std::thread> pool;
    for (int t = 0; t < threads; ++t)
      pool.emplace_back([&] {
        for (size_t i = 0; i < lines.size(); ++i) done += run_line(lines[i], (int)i + 1, true);
      });
    for (auto& th : pool) th.join();
    std::printf("threads %d commands %d failures %d launches %ld\n", threads, done.load(), g_fail.load(),
                stub_launches_total());
    return g_fail ? 1 : 0;
  }
  int done = 0;
  for (size_t i = 0; i < lines.size(); ++i) {
    const int before = g_fail;
    if (!run_line(lines[i], (int)i + 1, false)) continue;
    if (g_fail == before) std::printf("ok %d\n", (int)i + 1);
    ++done;
  }
  std::printf("commands %d failures %d launches %ld\n", done, g_fail.load(), stub_launches_total());
  return g_fail ? 1 : 0;
}
