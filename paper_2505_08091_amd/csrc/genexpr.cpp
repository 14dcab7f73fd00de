// Parser of the GenP expression language (grammar in genexpr.hpp).
#include "genexpr.hpp"

#include <cctype>
#include <stdexcept>

#include "layout.hpp"

namespace lego {

namespace {

GNodeP node(GNode::Kind k, std::vector<GNodeP> kids, i64 v = 0) {
  auto n = std::make_shared<GNode>();
  n->k = k;
  n->kids = std::move(kids);
  n->v = v;
  return n;
}
GNodeP num(i64 v) { return node(GNode::Num, {}, v); }
bool is_num(const GNodeP& n, i64* v) {
  if (n->k != GNode::Num) return false;
  *v = n->v;
  return true;
}

struct Parser {
  const std::string& s;
  const std::vector<std::string>& vars;
  const std::vector<std::pair<std::string, i64>>& consts;
  size_t p = 0;

  [[noreturn]] void fail(const std::string& what) const {
    throw std::invalid_argument("GenP expression, at offset " + std::to_string(p) + " of \"" + s + "\": " + what);
  }
  void ws() {
    while (p < s.size() && std::isspace((unsigned char)s[p])) ++p;
  }
  bool eat(const char* tok) {
    ws();
    size_t n = std::char_traits<char>::length(tok);
    if (s.compare(p, n, tok) != 0) return false;
    // keep '<' from eating the first half of '<<' or '<=' (and likewise)
    if (n == 1 && p + 1 < s.size()) {
      char a = tok[0], b = s[p + 1];
      if ((a == '<' || a == '>') && (b == '<' || b == '>' || b == '=')) return false;
      if ((a == '&' && b == '&') || (a == '|' && b == '|') || (a == '=' && b == '=') || (a == '!' && b == '='))
        return false;
    }
    p += n;
    return true;
  }
  void expect(const char* tok) {
    if (!eat(tok)) fail(std::string("expected '") + tok + "'");
  }

  GNodeP cond() {
    GNodeP c = lor();
    if (eat("?")) {
      GNodeP a = cond();
      expect(":");
      GNodeP b = cond();
      return node(GNode::Sel, {c, a, b});
    }
    return c;
  }
  GNodeP lor() {
    GNodeP a = land();
    while (eat("||")) a = node(GNode::Or, {a, land()});
    return a;
  }
  GNodeP land() {
    GNodeP a = bxor();
    while (eat("&&")) a = node(GNode::And, {a, bxor()});
    return a;
  }
  GNodeP bxor() {
    GNodeP a = band();
    while (eat("^")) a = node(GNode::Xor, {a, band()});
    return a;
  }
  GNodeP band() {
    GNodeP a = eq();
    while (eat("&")) {
      GNodeP b = eq();
      i64 m;
      if (!is_num(b, &m) || m < 0 || (m & (m + 1)) != 0) fail("'&' needs a constant mask 2^k - 1 on its right");
      a = node(GNode::Mod, {a}, m + 1);
    }
    return a;
  }
  GNodeP eq() {
    GNodeP a = rel();
    for (;;) {
      if (eat("=="))
        a = node(GNode::Eq, {a, rel()});
      else if (eat("!="))
        a = node(GNode::Not, {node(GNode::Eq, {a, rel()})});
      else
        return a;
    }
  }
  GNodeP rel() {
    GNodeP a = shift();
    for (;;) {
      if (eat("<=")) {  // a <= b  <=>  a < b + 1
        a = node(GNode::Lt, {a, node(GNode::Add, {shift(), num(1)})});
      } else if (eat(">=")) {  // a >= b  <=>  b < a + 1
        GNodeP b = shift();
        a = node(GNode::Lt, {b, node(GNode::Add, {a, num(1)})});
      } else if (eat("<")) {
        a = node(GNode::Lt, {a, shift()});
      } else if (eat(">")) {
        GNodeP b = shift();
        a = node(GNode::Lt, {b, a});
      } else {
        return a;
      }
    }
  }
  GNodeP shift() {
    GNodeP a = add();
    for (;;) {
      bool left = eat("<<");
      if (!left && !eat(">>")) return a;
      GNodeP b = add();
      i64 c;
      if (!is_num(b, &c) || c < 0 || c > 40) fail("shift amounts must be constants in [0, 40]");
      a = left ? node(GNode::Mul, {a, num(i64(1) << c)}) : node(GNode::Div, {a}, i64(1) << c);
    }
  }
  GNodeP add() {
    GNodeP a = mul();
    for (;;) {
      if (eat("+"))
        a = fold(node(GNode::Add, {a, mul()}));
      else if (eat("-"))
        a = fold(node(GNode::Sub, {a, mul()}));
      else
        return a;
    }
  }
  GNodeP mul() {
    GNodeP a = unary();
    for (;;) {
      if (eat("*")) {
        a = fold(node(GNode::Mul, {a, unary()}));
      } else if (eat("/") || eat("%")) {
        bool div = s[p - 1] == '/';
        GNodeP b = unary();
        i64 c;
        if (!is_num(b, &c) || c <= 0) fail("'/' and '%' need a positive constant divisor");
        a = fold(node(div ? GNode::Div : GNode::Mod, {a}, c));
      } else {
        return a;
      }
    }
  }
  GNodeP unary() {
    if (eat("-")) return fold(node(GNode::Neg, {unary()}));
    if (eat("!")) return node(GNode::Not, {unary()});
    return primary();
  }
  GNodeP primary() {
    ws();
    if (p >= s.size()) fail("unexpected end");
    if (std::isdigit((unsigned char)s[p])) {
      i64 v = 0;
      while (p < s.size() && std::isdigit((unsigned char)s[p])) {
        if (v > (i64(1) << 55)) fail("integer too large");
        v = v * 10 + (s[p++] - '0');
      }
      return num(v);
    }
    if (eat("(")) {
      GNodeP e = cond();
      expect(")");
      return e;
    }
    if (std::isalpha((unsigned char)s[p]) || s[p] == '_') {
      size_t b = p;
      while (p < s.size() && (std::isalnum((unsigned char)s[p]) || s[p] == '_')) ++p;
      std::string id = s.substr(b, p - b);
      if (id == "isqrt" || id == "min" || id == "max") {
        expect("(");
        std::vector<GNodeP> args = {cond()};
        while (eat(",")) args.push_back(cond());
        expect(")");
        if (id == "isqrt") {
          if (args.size() != 1) fail("isqrt takes one argument");
          return node(GNode::Isqrt, args);
        }
        if (args.size() != 2) fail(id + " takes two arguments");
        GNodeP lt = node(GNode::Lt, {args[0], args[1]});
        return id == "min" ? node(GNode::Sel, {lt, args[0], args[1]}) : node(GNode::Sel, {lt, args[1], args[0]});
      }
      for (size_t k = 0; k < vars.size(); ++k)
        if (vars[k] == id) {
          auto n = std::make_shared<GNode>();
          n->k = GNode::Var;
          n->var = (int)k;
          return n;
        }
      for (auto& c : consts)
        if (c.first == id) return num(c.second);
      fail("unknown name '" + id + "'");
    }
    fail(std::string("unexpected '") + s[p] + "'");
  }

  // Constant folding of arithmetic on literals (so divisors and shift amounts
  // may be written as expressions of the tile extents).
  GNodeP fold(GNodeP n) {
    i64 a, b;
    switch (n->k) {
      case GNode::Add:
        if (is_num(n->kids[0], &a) && is_num(n->kids[1], &b)) return num(a + b);
        break;
      case GNode::Sub:
        if (is_num(n->kids[0], &a) && is_num(n->kids[1], &b)) return num(a - b);
        break;
      case GNode::Mul:
        if (is_num(n->kids[0], &a) && is_num(n->kids[1], &b)) return num(a * b);
        break;
      case GNode::Div:
        if (is_num(n->kids[0], &a)) return num(IntAlg::fdiv_(a, n->v));
        break;
      case GNode::Mod:
        if (is_num(n->kids[0], &a)) return num(a - IntAlg::fdiv_(a, n->v) * n->v);
        break;
      case GNode::Neg:
        if (is_num(n->kids[0], &a)) return num(-a);
        break;
      default:
        break;
    }
    return n;
  }
};

}  // namespace

GNodeP parse_gexpr(const std::string& text, const std::vector<std::string>& vars,
                   const std::vector<std::pair<std::string, i64>>& consts) {
  Parser ps{text, vars, consts};
  GNodeP e = ps.cond();
  ps.ws();
  if (ps.p != text.size()) ps.fail("trailing text");
  return e;
}

}  // namespace lego
