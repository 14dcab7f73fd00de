// Lowering layouts to straight-line index code (Section IV-A).
//
// A lowering is built by a callback that declares variables in a Ctx and
// returns the output expressions.  It is run twice, with and without field
// refinement ("expanded" / "unexpanded"), and the variant with fewer operations
// is kept: the paper's cost model for pre-expansion.  Output is HIP C++ text
// using the LEGO_FN prelude macro, so the same text also compiles as host C++.
#pragma once

#include <functional>
#include <string>
#include <vector>

#include "expr.hpp"
#include "layout.hpp"

namespace lego {

struct FnSpec {
  std::vector<int> params;  // variable ids, in parameter order
  std::vector<Sum> outs;    // one or more outputs
  bool out_array = false;   // write outputs to one array parameter `o`
  bool valid = true;        // false: this variant cannot express the function
  // Optional: output k is known to lie in [0, out_bound[k]) (a layout's
  // inverse within its extents, its forward map within its physical size),
  // which lets 32-bit code compute it through out-of-range intermediates.
  std::vector<i64> out_bound;
  // The caller uses the outputs only modulo 2^32: they are parts of a sum
  // whose total lies in [0, 2^32), so 32-bit code may compute each part
  // through out-of-range values as long as it is right modulo 2^32.
  bool ring_out = false;
};

struct Emitted {
  std::string code;     // function definition text
  int ops = 0;          // operations in the chosen variant
  int ops_other = 0;    // operations in the other variant
  bool expanded = true;
  bool wide = false;    // 64-bit index type
};

std::string fn_text(const Ctx& c, const std::string& name, const FnSpec& f, bool force_wide, int* ops, bool* wide);

// Run `build` under both variants and emit the cheaper valid one.  Functions
// that are parts of one additive split must come from the same variant:
// `variant` = 0 forces the expanded form, 1 the unexpanded, -1 chooses.
Emitted emit_best(const std::string& name, const std::function<FnSpec(Ctx&)>& build, bool force_wide = false,
                  int variant = -1);

// out = L.apply(B^{-1}_{dims}(x)) for the logical flat index x.
FnSpec spec_apply_flat(Ctx& c, const Layout& l);
// out[k] = L.inv(p)[k] for the physical index p.
FnSpec spec_inv_flat(Ctx& c, const Layout& l);
// src = L_src.apply(L_dst.inv(p)) for the destination physical index p.
Sum remap_map(Ctx& c, const Layout& src, const Layout& dst, int p);
// The same map for an ExpandBy source without its -1 branch: returns the source
// position of destination position p assuming it is inside the original
// extents, and sets *valid to the 0/1 test that it is (1 for other sources).
Sum remap_map_masked(Ctx& c, const Layout& src, const Layout& dst, int p, Sum* valid);

// The common prelude of every generated source: index types, LEGO_FN and the
// helpers an expression may call (floor division of possibly negative values,
// an exact integer square root).
const char* prelude_text();

}  // namespace lego
