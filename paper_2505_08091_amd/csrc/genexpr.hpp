// User-defined GenP pieces written as integer expressions (Section III-B lets a
// GenP be any bijection f with its inverse f^-1; here both are given as text so
// they cross the C ABI and still lower to kernel code like the built-in ones).
//
// Grammar (C precedence and associativity, all values 64-bit integers):
//   expr    := cond
//   cond    := lor [ '?' expr ':' cond ]
//   lor     := land { '||' land }          C truth values, result 0/1
//   land    := bxor { '&&' bxor }          C truth values, result 0/1
//   bxor    := band { '^' band }           non-negative operands
//   band    := eq { '&' eq }               right operand a constant 2^k - 1
//   eq      := rel { ('==' | '!=') rel }
//   rel     := shift { ('<' | '<=' | '>' | '>=') shift }
//   shift   := add { ('<<' | '>>') add }   right operand a constant
//   add     := mul { ('+' | '-') mul }
//   mul     := unary { ('*' | '/' | '%') unary }   '/' '%' floor, by a positive constant
//   unary   := ('-' | '!') unary | primary
//   primary := integer | name | '(' expr ')' | func '(' expr { ',' expr } ')'
//   func    := isqrt (exact floor square root) | min | max
// Names: the coordinates i0 .. i{d-1} (also i, j, k for the first three) in the
// forward map, x in the inverse, and the tile extents n0 .. n{d-1} anywhere
// (constants).  Comparisons and logical operators give 0 or 1.  A GenP takes
// its forward result modulo the tile size and inverse coordinate k modulo n_k.
#pragma once

#include <memory>
#include <stdexcept>
#include <string>
#include <vector>

#include "expr.hpp"

namespace lego {

struct GNode;
using GNodeP = std::shared_ptr<const GNode>;

struct GNode {
  enum Kind { Num, Var, Add, Sub, Mul, Div, Mod, Xor, Lt, Eq, Sel, Isqrt, Neg, Not, And, Or } k;
  i64 v = 0;    // Num: value; Div/Mod: constant divisor
  int var = 0;  // Var: index into the environment
  std::vector<GNodeP> kids;
};

// Parses `text` over the variable names `vars` (their position is the Var
// index) with the constants `consts` (name -> value).  Throws
// std::invalid_argument with the offending position on a syntax error or on an
// operation the lowering cannot express (a non-constant divisor, a mask that is
// not 2^k - 1, ...).
GNodeP parse_gexpr(const std::string& text, const std::vector<std::string>& vars,
                   const std::vector<std::pair<std::string, i64>>& consts);

// The two sides of an expression GenP over dims n.
struct GenExpr {
  std::string apply_text;
  std::vector<std::string> inv_text;
  GNodeP apply;
  std::vector<GNodeP> inv;
};

// 1 when v != 0, else 0.
template <class A>
typename A::V truth(const A& al, const typename A::V& v) {
  return al.add(al.lt(al.c(0), v), al.lt(v, al.c(0)));
}

template <class A>
typename A::V eval_gexpr(const A& al, const GNode& g, const std::vector<typename A::V>& env) {
  using V = typename A::V;
  auto k = [&](size_t i) { return eval_gexpr(al, *g.kids[i], env); };
  switch (g.k) {
    case GNode::Num: return al.c(g.v);
    case GNode::Var: return env.at(g.var);
    case GNode::Add: return al.add(k(0), k(1));
    case GNode::Sub: return al.sub(k(0), k(1));
    case GNode::Mul: return al.mul(k(0), k(1));
    case GNode::Div: return al.div(k(0), g.v);
    case GNode::Mod: return al.mod(k(0), g.v);
    case GNode::Xor: return al.bxor(k(0), k(1));
    case GNode::Lt: return al.lt(k(0), k(1));
    case GNode::Eq: {
      V a = k(0), b = k(1);
      // a == b  <=>  !(a < b) && !(b < a)
      return al.mul(al.sub(al.c(1), al.lt(a, b)), al.sub(al.c(1), al.lt(b, a)));
    }
    case GNode::Sel: return al.sel(k(0), k(1), k(2));
    case GNode::Isqrt: return al.isqrt(k(0));
    case GNode::Neg: return al.sub(al.c(0), k(0));
    // C truth values: nonzero is true; the results are 0 or 1.
    case GNode::Not: return al.sub(al.c(1), truth(al, k(0)));
    case GNode::And: return al.mul(truth(al, k(0)), truth(al, k(1)));
    case GNode::Or: {
      V a = truth(al, k(0)), b = truth(al, k(1));
      return al.sub(al.add(a, b), al.mul(a, b));
    }
  }
  throw std::logic_error("bad expression node");
}

}  // namespace lego
