// Integer index-expression IR for lowering LEGO layouts to kernel code.
//
// The paper lowers a layout by evaluating its apply/inv on symbols and then
// simplifying floor-division and modulo with range information (Section IV-A,
// Table II).  Here every expression is kept in a canonical sum form
//
//     c0 + sum_t  c_t * atom_t
//
// where an atom is either a *digit field* of a variable, (v / a) % b (b == 0
// meaning "no modulo"), or an opaque operation (div, mod, product, xor, compare,
// select, integer sqrt) over sums.  Division and modulo by a constant n split a
// sum into the part whose coefficients are multiples of n and the remainder,
// refining digit fields at the boundary, and drop the remainder from the
// quotient when its proven range lies in [0, n): this is Table II's first five
// rules applied to mixed-radix digits, with interval analysis in place of the
// SMT-proved side conditions.  Adjacent fields of one variable are merged back
// (Table II's last rule, a*(x/a) + x%a -> x).  Layouts built from RegP pieces
// over power-of-two tiles therefore lower to shift-and-mask expressions with no
// division left and no lookup tables.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <vector>

namespace lego {

using i64 = long long;

struct Interval {
  i64 lo = 0, hi = 0;  // inclusive
};

struct Atom;
using AtomP = std::shared_ptr<const Atom>;

struct Term {
  i64 c;
  AtomP a;
};

struct Sum {
  i64 c0 = 0;
  std::vector<Term> t;  // canonical: sorted by atom key, distinct atoms, c != 0
  bool is_const() const { return t.empty(); }
};

enum class Op { Field, Div, Mod, Mul, Xor, Lt, Select, Isqrt };

struct Atom {
  Op op;
  int var = -1;  // Field
  i64 a = 1;     // Field divisor
  i64 b = 0;     // Field modulus (0: none)
  i64 k = 0;     // Div / Mod constant
  std::vector<Sum> kids;
  Interval r;
  std::string key;
};

// A lowering context: the variables and their ranges, and whether division and
// modulo may refine digit fields (the "expanded" form; the cost model compares
// both, as the paper does for pre-expansion).
struct Ctx {
  struct Var {
    std::string name;
    i64 hi;  // range [0, hi]
  };
  std::vector<Var> vars;
  bool expand = true;
  int var(const std::string& name, i64 extent);  // range [0, extent)
};

Sum cst(i64 v);
Sum var(const Ctx& c, int v);
Sum field(const Ctx& c, int v, i64 a, i64 b);
Sum add(const Ctx& c, const Sum& x, const Sum& y);
Sum sub(const Ctx& c, const Sum& x, const Sum& y);
Sum mulc(const Ctx& c, const Sum& x, i64 k);
Sum mul(const Ctx& c, const Sum& x, const Sum& y);
Sum fdiv(const Ctx& c, const Sum& x, i64 n);
Sum fmod(const Ctx& c, const Sum& x, i64 n);
Sum bxor(const Ctx& c, const Sum& x, const Sum& y);
Sum lt(const Ctx& c, const Sum& x, const Sum& y);          // 1 if x < y else 0
Sum select(const Ctx& c, const Sum& cond, const Sum& x, const Sum& y);  // cond ? x : y
Sum isqrt(const Ctx& c, const Sum& x);

Interval range(const Sum& s);
std::string key(const Sum& s);
bool depends_on(const Sum& s, int v);
// A positive divisor of every value s can take (from its constant, its
// coefficients and divisibility through mod, products and selects); 0 if s is
// identically zero.
i64 known_multiple(const Sum& s);
void vars_of(const Sum& s, std::vector<bool>& used);

// Replace variable v by an expression.
Sum subst(const Ctx& c, const Sum& s, int v, const Sum& repl);

// Split s into the terms that depend on any variable in `group` and the rest.
// Returns false when some atom depends on variables both in and outside the
// group (the expression is not additively separable).
bool split_by(const Sum& s, const std::vector<int>& group, Sum* in_group, Sum* rest);

// Digit structure of a pure field sum: no constant, every atom a Field of one
// variable with a positive weight, and the fields of that variable tile its
// digits without overlap.
struct Digit {
  i64 a, b, coeff;  // (v / a) % b contributes coeff * digit
};
bool digits_of(const Ctx& c, const Sum& s, int v, std::vector<Digit>* out);

// Printing.  The index type is 32-bit unsigned when every printed quantity is
// proven to lie in [0, 2^32), 64-bit signed otherwise.
struct Printed {
  std::string text;
  int ops = 0;
  bool wide = false;
};
Printed print(const Ctx& c, const Sum& s);
// Several outputs printed with shared common subexpressions bound in `lets`.
struct PrintedMany {
  std::vector<std::string> outs;
  std::string lets;
  int ops = 0;
};
PrintedMany print_many(const Ctx& c, const std::vector<Sum>& outs, bool wide);
// 32-bit index code evaluates s exactly (fits32), or congruently modulo 2^32
// (ring32: exact wherever the value is known to lie in [0, 2^32)).
bool fits32(const Sum& s);
bool ring32(const Sum& s);

}  // namespace lego
