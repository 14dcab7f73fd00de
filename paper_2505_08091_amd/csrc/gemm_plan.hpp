// GEMM planning: a lego_gemm_desc becomes one generated kernel whose every
// index expression is lowered from a layout.
#pragma once

#include <functional>
#include <memory>
#include <string>
#include <utility>
#include <vector>

#include "lego.h"
#include "layout.hpp"
#include "plans.hpp"

namespace lego {

struct GemmRequest {
  i64 M = 0, N = 0, K = 0;
  int dtype = LEGO_BF16;
  int bm = 0, bn = 0, bk = 0, wm = 0, wn = 0, group_m = 0, xcd = 0;
  int stages = 0;  // LDS stages; 0: chosen
  LayoutP a, b, c, sched, lds_a, lds_b;  // null: defaults
  LayoutP frag_a, frag_b, frag_c;        // null: chosen; else they select the MFMA instruction
};

struct GemmPlan : KernelPlan {
  // direct global-to-LDS copies whose 128x128 wave tiles fit the registers
  // (not transposing reads with padded tiles)
  bool wide_ok = false;
};

GemmRequest gemm_request(const lego_gemm_desc& d, const std::function<LayoutP(lego_layout_t)>& resolve);
std::shared_ptr<GemmPlan> gemm_plan_cached(const GemmRequest& rq);
GemmPlan plan_gemm(const GemmRequest& rq);

// MFMA fragment layouts (instr 0: 32x32x16, 1: 16x16x32; operand 0 A, 1 B,
// 2 C/D): logical (lane, element) -> row * cols + col inside the block.
LayoutP mfma_fragment_layout(int instr, int operand);

// Generated sources for the built-in configurations (name, source).
std::vector<std::pair<std::string, std::string>> selftest_sources();

}  // namespace lego
