// Rule text -> typed rules -> strata -> per-rule join plans.  Host-only.
//
// Accepted subset of the paper's surface syntax (Sec. 3.1, 3.3, 3.5):
//   rule    := head ':-' literal (',' literal)* '.'
//   head    := name '(' Var (',' Var)* [',' agg '(' Var ')'] ')'
//   literal := name '(' term (',' term)* ')'
//            | Var 'is' term (('+' | '-') term)*
//            | term cmp term            cmp in != == < <= > >=
//   term    := Var | '_' | integer | float
// Variables start with an upper-case letter or '_'; '//' starts a comment.
#include <algorithm>
#include <cctype>
#include <cstring>
#include <functional>
#include <set>
#include <sstream>

#include "engine.h"

namespace xlh {

const char* agg_name(Agg a) {
  switch (a) {
    case Agg::COUNT: return "count";
    case Agg::SUM: return "sum";
    case Agg::MIN: return "min";
    case Agg::MAX: return "max";
    case Agg::LSE: return "logsumexp";
    default: return "set";
  }
}

namespace {

struct Tok {
  enum Kind { NAME, NUM, OP, END } kind;
  std::string s;
  int line;
};

struct Lexer {
  std::vector<Tok> toks;
  std::string err;
  bool run(const char* text) {
    int line = 1;
    const char* p = text;
    while (*p) {
      if (*p == '\n') { ++line; ++p; continue; }
      if (isspace((unsigned char)*p)) { ++p; continue; }
      if (p[0] == '/' && p[1] == '/') { while (*p && *p != '\n') ++p; continue; }
      if (isalpha((unsigned char)*p) || *p == '_') {
        const char* b = p;
        while (isalnum((unsigned char)*p) || *p == '_') ++p;
        toks.push_back({Tok::NAME, std::string(b, p), line});
        continue;
      }
      if (isdigit((unsigned char)*p)) {
        const char* b = p;
        while (isdigit((unsigned char)*p)) ++p;
        if (*p == '.' && isdigit((unsigned char)p[1])) {
          ++p;
          while (isdigit((unsigned char)*p)) ++p;
        }
        if (*p == 'e' || *p == 'E') {
          const char* q = p + 1;
          if (*q == '+' || *q == '-') ++q;
          if (isdigit((unsigned char)*q)) {
            p = q;
            while (isdigit((unsigned char)*p)) ++p;
          }
        }
        toks.push_back({Tok::NUM, std::string(b, p), line});
        continue;
      }
      static const char* ops2[] = {":-", "!=", "==", "<=", ">="};
      bool two = false;
      for (const char* o : ops2)
        if (p[0] == o[0] && p[1] == o[1]) {
          toks.push_back({Tok::OP, std::string(o), line});
          p += 2;
          two = true;
          break;
        }
      if (two) continue;
      if (strchr("(),.+-<>", *p)) {
        toks.push_back({Tok::OP, std::string(1, *p), line});
        ++p;
        continue;
      }
      err = "line " + std::to_string(line) + ": unexpected character '" + std::string(1, *p) + "'";
      return false;
    }
    toks.push_back({Tok::END, "", line});
    return true;
  }
};

bool is_var_name(const std::string& s) { return !s.empty() && (isupper((unsigned char)s[0]) || s[0] == '_'); }

struct Parser {
  std::vector<Tok>& t;
  size_t i = 0;
  std::string err;
  explicit Parser(std::vector<Tok>& tt) : t(tt) {}

  bool fail(const std::string& m) {
    if (err.empty()) err = "line " + std::to_string(t[i].line) + ": " + m;
    return false;
  }
  bool expect(const char* s) {
    if (t[i].s == s && t[i].kind != Tok::END) { ++i; return true; }
    return fail(std::string("expected '") + s + "' but found '" + t[i].s + "'");
  }
  bool term(Term* out) {
    bool neg = false;
    if (t[i].kind == Tok::OP && t[i].s == "-" && t[i + 1].kind == Tok::NUM) { neg = true; ++i; }
    const Tok& k = t[i];
    if (k.kind == Tok::NUM) {
      ++i;
      if (k.s.find_first_of(".eE") != std::string::npos) {
        out->kind = Term::FLOAT;
        out->fval = strtod(k.s.c_str(), nullptr) * (neg ? -1.0 : 1.0);
      } else {
        out->kind = Term::INT;
        errno = 0;
        const unsigned long long u = strtoull(k.s.c_str(), nullptr, 10);
        if (errno == ERANGE || (neg && u > (1ull << 63))) return fail("integer constant outside the 64-bit range");
        out->ival = neg ? (int64_t)(0ull - u) : (int64_t)u;
        out->big = !neg && u > (unsigned long long)INT64_MAX;
      }
      return true;
    }
    if (k.kind == Tok::NAME) {
      ++i;
      if (k.s == "_") { out->kind = Term::ANON; return true; }
      if (is_var_name(k.s)) { out->kind = Term::VAR; out->name = k.s; return true; }
      return fail("expected a variable or constant, found '" + k.s + "'");
    }
    return fail("expected a term, found '" + k.s + "'");
  }
  static Agg agg_of(const std::string& s) {
    if (s == "count") return Agg::COUNT;
    if (s == "sum") return Agg::SUM;
    if (s == "min") return Agg::MIN;
    if (s == "max") return Agg::MAX;
    if (s == "logsumexp") return Agg::LSE;
    return Agg::NONE;
  }
  bool rule(RuleAst* r) {
    size_t start = i;
    if (t[i].kind != Tok::NAME || is_var_name(t[i].s)) return fail("expected a rule head");
    r->head = t[i++].s;
    if (!expect("(")) return false;
    while (true) {
      Agg a = t[i].kind == Tok::NAME ? agg_of(t[i].s) : Agg::NONE;
      if (a != Agg::NONE && t[i + 1].s == "(") {
        if (r->agg != Agg::NONE) return fail("at most one aggregate per head");
        r->agg = a;
        i += 2;
        Term v;
        if (!term(&v)) return false;
        if (v.kind != Term::VAR) return fail("an aggregate takes one variable");
        r->agg_var = v.name;
        if (!expect(")")) return false;
      } else {
        if (r->agg != Agg::NONE) return fail("the aggregate must be the last head argument");
        Term v;
        if (!term(&v)) return false;
        r->head_args.push_back(v);
      }
      if (t[i].s == ")") { ++i; break; }
      if (!expect(",")) return false;
    }
    if (t[i].s == ".") return fail("facts are not accepted in rule text; load them as relation rows");
    if (!expect(":-")) return false;
    while (true) {
      const bool negated = t[i].kind == Tok::NAME && t[i].s == "not" && t[i + 1].kind == Tok::NAME &&
                           !is_var_name(t[i + 1].s) && t[i + 2].s == "(";
      if (negated) ++i;
      if (t[i].kind == Tok::NAME && !is_var_name(t[i].s) && t[i + 1].s == "(") {
        AtomAst a;
        a.pred = t[i].s;
        i += 2;
        while (true) {
          Term v;
          if (!term(&v)) return false;
          a.args.push_back(v);
          if (t[i].s == ")") { ++i; break; }
          if (!expect(",")) return false;
        }
        (negated ? r->negs : r->atoms).push_back(a);
      } else if (t[i].kind == Tok::NAME && t[i + 1].kind == Tok::NAME && t[i + 1].s == "is") {
        if (!is_var_name(t[i].s) || t[i].s == "_") return fail("the left side of 'is' must be a variable");
        RuleAst::Assign as;
        as.var = t[i].s;
        i += 2;
        Term v;
        if (!term(&v)) return false;
        as.parts.push_back({1, v});
        while (t[i].kind == Tok::OP && (t[i].s == "+" || t[i].s == "-")) {
          int sign = t[i].s == "+" ? 1 : -1;
          ++i;
          if (!term(&v)) return false;
          as.parts.push_back({sign, v});
        }
        r->assigns.push_back(as);
      } else {
        RuleAst::Cmp c;
        if (!term(&c.lhs)) return false;
        static const char* names[] = {"!=", "==", "<", "<=", ">", ">="};
        int op = -1;
        for (int k = 0; k < 6; ++k)
          if (t[i].s == names[k]) op = k;
        if (op < 0) return fail("expected a comparison operator, found '" + t[i].s + "'");
        ++i;
        c.op = op;
        if (!term(&c.rhs)) return false;
        r->cmps.push_back(c);
      }
      if (t[i].s == ".") { ++i; break; }
      if (!expect(",")) return false;
    }
    std::ostringstream os;
    for (size_t k = start; k < i; ++k) os << t[k].s << (k + 1 < i && t[k].kind == Tok::NAME && t[k + 1].kind == Tok::NAME ? " " : "");
    r->text = os.str();
    return true;
  }
};

// ------------------------------------------------------------------ planning
// The triangle shape (see RulePlan::wcoj): a set head over three distinct
// variables h0, h1, h2 and exactly three body atoms, each over a binary int32
// relation with two of the variables, one atom per pair.
static bool triangle_plan(Context* ctx, const RuleAst& r, RulePlan* p) {
  if (r.head_args.size() != 3 || r.agg != Agg::NONE || r.atoms.size() != 3 || !r.negs.empty() ||
      !r.assigns.empty() || !r.cmps.empty())
    return false;
  std::string hv[3];
  for (int j = 0; j < 3; ++j) {
    if (r.head_args[j].kind != Term::VAR) return false;
    hv[j] = r.head_args[j].name;
  }
  if (hv[0] == hv[1] || hv[1] == hv[2] || hv[0] == hv[2]) return false;
  auto var_index = [&](const Term& t) {
    if (t.kind != Term::VAR) return -1;
    for (int j = 0; j < 3; ++j)
      if (t.name == hv[j]) return j;
    return -1;
  };
  // atom covering head variables {u, v}: its relation and the columns of u, v
  Relation* rel[3] = {nullptr, nullptr, nullptr};
  int col[3][2] = {};
  const int pu[3] = {0, 1, 0}, pv[3] = {1, 2, 2};  // pairs (h0,h1), (h1,h2), (h0,h2)
  for (const AtomAst& a : r.atoms) {
    Relation* q = ctx->find(a.pred);
    if (!q || q->arity != 2 || q->types[0] != T_I32 || q->types[1] != T_I32) return false;
    const int i0 = var_index(a.args[0]), i1 = var_index(a.args[1]);
    if (i0 < 0 || i1 < 0 || i0 == i1) return false;
    const int lo = std::min(i0, i1), hi = std::max(i0, i1);
    int k = -1;
    for (int m = 0; m < 3; ++m)
      if (pu[m] == lo && pv[m] == hi) k = m;
    if (k < 0 || rel[k]) return false;
    rel[k] = q;
    col[k][0] = i0 == lo ? 0 : 1;  // column of the pair's first variable
    col[k][1] = 1 - col[k][0];
  }
  p->wcoj = true;
  p->head = ctx->find(r.head);
  p->driver = rel[0];
  p->tri_a[0] = col[0][0];  // X
  p->tri_a[1] = col[0][1];  // Y
  p->tri_brel = rel[1];
  p->tri_b[0] = col[1][0];  // Y
  p->tri_b[1] = col[1][1];  // Z
  p->tri_crel = rel[2];
  p->tri_c[0] = col[2][0];  // X
  p->tri_c[1] = col[2][1];  // Z
  p->nkey = 3;
  return true;
}

struct Planner {
  Context* ctx;
  std::string err;
  xl_status status = XL_OK;

  bool fail(xl_status st, const std::string& m) {
    if (status == XL_OK) { status = st; err = m; }
    return false;
  }

  static int natural_type(const Term& t) { return t.kind == Term::FLOAT ? XL_F32 : XL_I32; }
  // Stored image of constant t in a column of type lt; false when t is not a
  // value of lt.  The 8-byte types get their image (a dictionary rank) when
  // a run starts: *wide is set and *key receives the value's order key.
  static bool const_image(const Term& t, int lt, uint32_t* bits, bool* wide, unsigned long long* key) {
    *wide = false;
    *bits = 0;
    *key = 0;
    if (t.kind == Term::FLOAT) {
      if (lt == XL_F32) {
        const float f = (float)t.fval;
        memcpy(bits, &f, 4);
        return true;
      }
      if (lt != XL_F64) return false;
      unsigned long long b;
      memcpy(&b, &t.fval, 8);
      *key = order_key64(b, XL_F64);
      *wide = true;
      return true;
    }
    if (t.kind != Term::INT) return false;
    const int64_t v = t.ival;
    switch (lt) {
      case XL_I32:
        if (t.big || v < INT32_MIN || v > INT32_MAX) return false;
        *bits = (uint32_t)(int32_t)v;
        return true;
      case XL_U32:
        if (t.big || v < 0 || v > (int64_t)UINT32_MAX) return false;
        *bits = (uint32_t)v ^ 0x80000000u;
        return true;
      case XL_BOOL:
        if (t.big || (v != 0 && v != 1)) return false;
        *bits = (uint32_t)v;
        return true;
      case XL_I64:
        if (t.big) return false;
        *key = order_key64((unsigned long long)v, XL_I64);
        *wide = true;
        return true;
      case XL_U64:
        if (!t.big && v < 0) return false;
        *key = (unsigned long long)v;
        *wide = true;
        return true;
      default:
        return false;
    }
  }

  // Plan one rule with atom `drv` scanned first.
  bool plan(const RuleAst& r, int rule_id, int drv, bool delta, RulePlan* out) {
    RulePlan p;
    p.rule = rule_id;
    p.head = ctx->find(r.head);
    std::map<std::string, int> slot;
    std::map<std::string, int> vtype;  // declared (xl_type) type of each variable
    std::map<std::string, int> bstage;  // binding stage (0 = driver, k+1 = step k)
    std::set<std::string> assigned;
    for (auto& a : r.assigns) {
      if (assigned.count(a.var)) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': " + a.var + " is assigned twice");
      assigned.insert(a.var);
    }
    auto new_slot = [&](const std::string& v) -> int {
      auto it = slot.find(v);
      if (it != slot.end()) return it->second;
      int s = (int)slot.size();
      slot[v] = s;
      return s;
    };
    // step: the join step the atom becomes (-1 for the driver)
    auto bind_atom = [&](const AtomAst& a, Relation* rel, int stage, int key_col, ColAct* act, int step) -> bool {
      for (int j = 0; j < rel->arity; ++j) {
        const Term& t = a.args[j];
        ColAct c{};
        c.type = rel->types[j];
        if (j == key_col) {
          act[j] = c;
          continue;
        }
        if (t.kind == Term::ANON) {
          c.kind = CA_NONE;
        } else if (t.kind == Term::INT || t.kind == Term::FLOAT) {
          bool wide;
          unsigned long long key;
          if (!const_image(t, rel->ltypes[j], &c.cval, &wide, &key))
            return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': constant is not a " + type_name(rel->ltypes[j]) +
                                              " value (column " + std::to_string(j) + " of " + rel->name + ")");
          c.kind = CA_CHECK_CONST;
          if (wide)
            p.wconsts.push_back(step < 0 ? WideConst{0, rel->ltypes[j], (int16_t)j, 0, key}
                                         : WideConst{1, rel->ltypes[j], (int16_t)step, (int16_t)j, key});
        } else {
          if (assigned.count(t.name))
            return fail(XL_UNSUPPORTED, "rule '" + r.text + "': " + t.name + " is both an 'is' result and an atom argument");
          auto vt = vtype.find(t.name);
          if (vt != vtype.end() && vt->second != rel->ltypes[j])
            return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': variable " + t.name + " is used at two column types");
          if (bstage.count(t.name)) {
            c.kind = CA_CHECK_SLOT;
            c.slot = (int8_t)slot[t.name];
          } else {
            c.kind = CA_BIND;
            c.slot = (int8_t)new_slot(t.name);
            bstage[t.name] = stage;
            vtype[t.name] = rel->ltypes[j];
          }
          p.var_sources[slot[t.name]].push_back({rel, j});
        }
        act[j] = c;
      }
      return true;
    };

    // driver
    const AtomAst& da = r.atoms[drv];
    p.driver = ctx->find(da.pred);
    p.driver_delta = delta;
    if (!bind_atom(da, p.driver, 0, -1, p.driver_act, -1)) return false;
    // join order: first remaining atom that shares a bound variable
    std::vector<int> rest;
    for (int k = 0; k < (int)r.atoms.size(); ++k)
      if (k != drv) rest.push_back(k);
    while (!rest.empty()) {
      int pick = -1, key_col = -1;
      for (size_t q = 0; q < rest.size() && pick < 0; ++q) {
        const AtomAst& a = r.atoms[rest[q]];
        Relation* rel = ctx->find(a.pred);
        for (int j = 0; j < rel->arity; ++j) {
          const Term& t = a.args[j];
          if (t.kind == Term::VAR && bstage.count(t.name) && rel->types[j] == T_I32) {
            pick = (int)q;
            key_col = j;
            break;
          }
        }
      }
      if (pick < 0)
        return fail(XL_UNSUPPORTED, "rule '" + r.text + "': an atom shares no bound int32 variable with the atoms before it (cross products are not supported)");
      const AtomAst& a = r.atoms[rest[pick]];
      StepPlan st;
      st.rel = ctx->find(a.pred);
      st.key_col = key_col;
      const std::string& kv = a.args[key_col].name;
      if (vtype[kv] != st.rel->ltypes[key_col])
        return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': join variable " + kv + " is used at two column types");
      st.key_slot = slot[kv];
      p.var_sources[st.key_slot].push_back({st.rel, key_col});
      int stage = (int)p.steps.size() + 1;
      if (!bind_atom(a, st.rel, stage, key_col, st.act, (int)p.steps.size())) return false;
      p.steps.push_back(st);
      rest.erase(rest.begin() + pick);
    }
    const int nst = (int)p.steps.size();
    const int nkst = nst > 0 ? nst : 1;  // kernel stages
    p.stage_ops.assign(nkst, {});
    p.stage_consts.assign(nkst, {});
    auto kstage_of = [&](int bind_stage) { return bind_stage > 0 ? bind_stage - 1 : 0; };
    std::map<std::string, int> avail;  // var -> kernel stage where available
    for (auto& kv : bstage) avail[kv.first] = kstage_of(kv.second);

    // declared type of a term in an expression: a bound variable's, or 0 for
    // a constant (typed by the other operand)
    auto term_type = [&](const Term& t, int* lt) -> bool {
      *lt = 0;
      if (t.kind == Term::ANON) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': '_' cannot be used in arithmetic or comparisons");
      if (t.kind != Term::VAR) return true;
      if (!avail.count(t.name)) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': " + t.name + " is not bound before it is used");
      *lt = vtype[t.name];
      return true;
    };
    // operand encoding of t at type lt (a constant becomes a stage constant)
    auto operand = [&](int ks, const Term& t, int lt, int8_t* enc) -> bool {
      if (t.kind == Term::VAR) {
        *enc = (int8_t)slot[t.name];
        return true;
      }
      auto& cs = p.stage_consts[ks];
      if (cs.size() >= (size_t)MAXK) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': too many constants");
      uint32_t bits;
      bool wide;
      unsigned long long key;
      if (!const_image(t, lt, &bits, &wide, &key))
        return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': a constant is not a " + type_name(lt) + " value");
      if (wide) p.wconsts.push_back(WideConst{2, (uint8_t)lt, (int16_t)ks, (int16_t)cs.size(), key});
      cs.push_back(bits);
      *enc = (int8_t)(-(int)cs.size());
      return true;
    };
    auto stage_needed = [&](const std::vector<const Term*>& ts) -> int {
      int s = 0;
      for (const Term* t : ts)
        if (t->kind == Term::VAR && avail.count(t->name)) s = std::max(s, avail[t->name]);
      return s;
    };
    for (auto& as : r.assigns) {
      std::vector<const Term*> ts;
      for (auto& pt : as.parts) ts.push_back(&pt.second);
      int ks = stage_needed(ts);
      int s = new_slot(as.var);
      // the type of the first variable operand, else of the first constant
      int ty = 0;
      for (auto& pt : as.parts) {
        int t1;
        if (!term_type(pt.second, &t1)) return false;
        if (!ty) ty = t1;
      }
      if (!ty) ty = natural_type(as.parts[0].second);
      if (ty != XL_I32 && ty != XL_F32)
        return fail(XL_UNSUPPORTED, "rule '" + r.text + "': arithmetic on " + type_name(ty) + " values is not supported");
      for (size_t q = 0; q < as.parts.size(); ++q) {
        int t1;
        int8_t e1;
        (void)term_type(as.parts[q].second, &t1);
        if ((t1 && t1 != ty) || (!t1 && natural_type(as.parts[q].second) != ty))
          return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': 'is' mixes int32 and float32 operands");
        if (!operand(ks, as.parts[q].second, ty, &e1)) return false;
        MicroOp op{};
        op.type = phys_type(ty);
        op.dst = (int8_t)s;
        if (q == 0) {
          if (as.parts[0].first > 0) {
            op.kind = OP_MOV;
            op.a = e1;
          } else {  // 0 - x
            Term zero;
            zero.kind = ty == XL_F32 ? Term::FLOAT : Term::INT;
            int8_t ez;
            if (!operand(ks, zero, ty, &ez)) return false;
            op.kind = OP_SUB;
            op.a = ez;
            op.b = e1;
          }
        } else {
          op.kind = as.parts[q].first > 0 ? OP_ADD : OP_SUB;
          op.a = (int8_t)s;
          op.b = e1;
        }
        p.stage_ops[ks].push_back(op);
      }
      vtype[as.var] = ty;
      avail[as.var] = ks;
      p.var_is_arith[s] = true;
    }
    for (auto& c : r.cmps) {
      int ks = stage_needed({&c.lhs, &c.rhs});
      MicroOp op{};
      op.kind = OP_CMP;
      op.cmp = (uint8_t)c.op;
      int t1, t2;
      if (!term_type(c.lhs, &t1) || !term_type(c.rhs, &t2)) return false;
      if (!t1 && !t2) {  // two constants: their natural types
        t1 = natural_type(c.lhs);
        t2 = natural_type(c.rhs);
      }
      if (t1 && t2 && t1 != t2)
        return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': comparison between " + type_name(t1) + " and " + type_name(t2));
      const int lt = t1 ? t1 : t2;
      if (!operand(ks, c.lhs, lt, &op.a) || !operand(ks, c.rhs, lt, &op.b)) return false;
      op.type = phys_type(lt);
      p.stage_ops[ks].push_back(op);
    }
    // negated literals: a membership test at the first stage where all their
    // variables are bound
    if (r.negs.size() > (size_t)MAXNEG)
      return fail(XL_UNSUPPORTED, "rule '" + r.text + "': at most " + std::to_string(MAXNEG) + " negated literals");
    for (const AtomAst& a : r.negs) {
      Relation* rel = ctx->find(a.pred);
      NegPlan np;
      np.rel = rel;
      std::vector<const Term*> used;
      std::vector<int> cols;
      for (int j = 0; j < rel->arity; ++j) {
        const Term& t = a.args[j];
        if (t.kind == Term::ANON) continue;
        if (t.kind == Term::VAR) {
          if (!avail.count(t.name))
            return fail(XL_UNSUPPORTED, "rule '" + r.text + "': " + t.name + " occurs in 'not " + a.pred +
                                            "' but in no positive atom or 'is' before it");
          if (vtype[t.name] != rel->ltypes[j])
            return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': variable " + t.name + " is used at two column types");
        }
        if (rel->types[j] != T_I32)
          return fail(XL_UNSUPPORTED, "rule '" + r.text + "': negated literals may not constrain float32 columns");
        used.push_back(&t);
        cols.push_back(j);
      }
      // (a variable may occur twice: the packed key then asks for a row with
      // both columns equal to it)
      if (used.size() > 2)
        return fail(XL_UNSUPPORTED, "rule '" + r.text + "': 'not " + a.pred + "' constrains more than two columns");
      np.ncols = (int)used.size();
      for (int q = 0; q < np.ncols; ++q) np.col[q] = cols[q];
      const int ks = stage_needed(used);
      MicroOp op{};
      op.kind = OP_NOTIN;
      op.cmp = (uint8_t)p.negs.size();
      op.type = (uint8_t)np.ncols;
      op.a = 0;
      op.b = 0;
      if (np.ncols > 0 && !operand(ks, *used[0], rel->ltypes[cols[0]], &op.a)) return false;
      if (np.ncols > 1 && !operand(ks, *used[1], rel->ltypes[cols[1]], &op.b)) return false;
      p.stage_ops[ks].push_back(op);
      p.negs.push_back(np);
    }
    if ((int)slot.size() > MAXV) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': more than 8 variables");
    for (int k = 0; k < nkst; ++k)
      if (p.stage_ops[k].size() > (size_t)MAXOPS) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': too many comparisons/arithmetic terms");

    // head
    Relation* h = p.head;
    const int nkey = (int)r.head_args.size();
    p.nkey = nkey;
    for (int j = 0; j < nkey; ++j) {
      const Term& t = r.head_args[j];
      if (t.kind != Term::VAR) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': head arguments must be variables");
      if (!avail.count(t.name)) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': head variable " + t.name + " does not occur in the body");
      if (vtype[t.name] != h->ltypes[j]) return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': head argument " + t.name + " does not match column " + std::to_string(j) + " of " + h->name);
      p.key_slot[j] = slot[t.name];
    }
    if (r.agg != Agg::NONE) {
      if (!avail.count(r.agg_var)) return fail(XL_UNSUPPORTED, "rule '" + r.text + "': aggregated variable " + r.agg_var + " does not occur in the body");
      const int vt = h->ltypes[nkey];
      if (r.agg == Agg::COUNT) {
        if (vt != XL_I32) return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': count produces an int32 column");
        p.val_slot = -1;
      } else {
        if (vtype[r.agg_var] != vt) return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': aggregated variable does not match the head's value column");
        if (r.agg == Agg::LSE && vt != XL_F32) return fail(XL_TYPE_MISMATCH, "rule '" + r.text + "': logsumexp needs a float32 column");
        if (r.agg == Agg::SUM && vt != XL_I32 && vt != XL_F32)
          return fail(XL_UNSUPPORTED, "rule '" + r.text + "': sum over " + type_name(vt) + " values is not supported");
        p.val_slot = slot[r.agg_var];
      }
      p.val_type = phys_type(vt);
    }
    // live slots between kernel stages
    p.live_after.assign(nkst, {});
    for (int k = 0; k + 1 < nkst; ++k) {
      std::set<int> used;
      for (int q = k + 1; q < nst; ++q) {
        used.insert(p.steps[q].key_slot);
        for (int j = 0; j < p.steps[q].rel->arity; ++j)
          if (p.steps[q].act[j].kind == CA_CHECK_SLOT) used.insert(p.steps[q].act[j].slot);
      }
      for (int q = k + 1; q < nkst; ++q)
        for (auto& op : p.stage_ops[q]) {
          if (op.kind == OP_MOV || op.kind == OP_ADD || op.kind == OP_SUB || op.kind == OP_CMP) {
            if (op.a >= 0) used.insert(op.a);
            if (op.kind != OP_MOV && op.b >= 0) used.insert(op.b);
          }
        }
      for (int j = 0; j < nkey; ++j) used.insert(p.key_slot[j]);
      if (p.val_slot >= 0) used.insert(p.val_slot);
      for (auto& kv : avail)
        if (kv.second <= k && used.count(slot[kv.first])) p.live_after[k].push_back(slot[kv.first]);
      std::sort(p.live_after[k].begin(), p.live_after[k].end());
    }
    // transitive-closure shape (see RulePlan::carried)
    if (delta && p.driver == p.head && p.head->arity == 2 && r.agg == Agg::NONE && nst == 1 &&
        p.steps[0].rel != p.head &&
        p.stage_ops[0].empty() && p.driver_act[0].kind == CA_BIND && p.driver_act[1].kind == CA_BIND &&
        p.driver_act[0].slot != p.driver_act[1].slot && p.steps[0].key_slot == p.driver_act[1].slot &&
        p.key_slot[0] == p.driver_act[0].slot) {
      int ycol = -1, nbind = 0, nother = 0;
      for (int j = 0; j < p.steps[0].rel->arity; ++j) {
        if (j == p.steps[0].key_col) continue;
        if (p.steps[0].act[j].kind == CA_BIND) { ++nbind; ycol = j; }
        else if (p.steps[0].act[j].kind != CA_NONE) ++nother;
      }
      if (nbind == 1 && nother == 0 && p.steps[0].act[ycol].slot == p.key_slot[1] &&
          p.steps[0].rel->types[ycol] == T_I32) {
        p.carried = true;
        p.carried_ycol = ycol;
      }
    }
    // carried value shape (see RulePlan::carried_val)
    if (delta && p.negs.empty() && p.driver == p.head && p.head->arity == 3 &&
        (r.agg == Agg::SUM || r.agg == Agg::LSE || r.agg == Agg::MIN || r.agg == Agg::MAX) &&
        nst == 1 && p.steps[0].rel != p.head && p.driver_act[0].kind == CA_BIND && p.driver_act[1].kind == CA_BIND &&
        (p.driver_act[2].kind == CA_BIND || p.driver_act[2].kind == CA_NONE) &&
        p.driver_act[0].slot != p.driver_act[1].slot && p.steps[0].key_slot == p.driver_act[1].slot &&
        p.key_slot[0] == p.driver_act[0].slot && p.val_slot >= 0) {
      int ycol = -1;
      for (int j = 0; j < p.steps[0].rel->arity; ++j)
        if (j != p.steps[0].key_col && p.steps[0].act[j].kind == CA_BIND && p.steps[0].act[j].slot == p.key_slot[1])
          ycol = j;
      if (ycol >= 0 && p.steps[0].rel->types[ycol] == T_I32) {
        p.carried_val = true;
        p.carried_ycol = ycol;
        p.cv_slot_s = p.driver_act[0].slot;
        p.cv_slot_z = p.driver_act[1].slot;
        p.cv_slot_p = p.driver_act[2].kind == CA_BIND ? p.driver_act[2].slot : -1;
      }
    }
    *out = p;
    return true;
  }
};

}  // namespace

xl_status compile_program(Context* ctx, const char* text, Program** out) {
  Lexer lx;
  if (!lx.run(text)) return ctx->fail(XL_PARSE_ERROR, lx.err);
  Parser ps(lx.toks);
  auto prog = new Program();
  prog->ctx = ctx;
  while (lx.toks[ps.i].kind != Tok::END) {
    RuleAst r;
    if (!ps.rule(&r)) {
      delete prog;
      return ctx->fail(XL_PARSE_ERROR, ps.err);
    }
    prog->rules.push_back(r);
  }
  auto bad = [&](xl_status st, const std::string& m) {
    delete prog;
    return ctx->fail(st, m);
  };
  if (prog->rules.empty()) return bad(XL_INVALID_ARGUMENT, "no rules");
  // declarations, arity, head kinds
  for (auto& r : prog->rules) {
    Relation* h = ctx->find(r.head);
    if (!h) return bad(XL_INVALID_ARGUMENT, "relation '" + r.head + "' is not declared");
    const int want = (int)r.head_args.size() + (r.agg != Agg::NONE ? 1 : 0);
    if (want != h->arity) return bad(XL_INVALID_ARGUMENT, "rule '" + r.text + "': head has " + std::to_string(want) + " arguments but " + h->name + " has arity " + std::to_string(h->arity));
    RulePlan tri;
    if (r.head_args.empty() || (r.head_args.size() > 2 && !triangle_plan(ctx, r, &tri)))
      return bad(XL_UNSUPPORTED, "rule '" + r.text + "': derived relations need one or two key columns "
                                 "(three only for a triangle join h(X,Y,Z) :- a(X,Y), b(Y,Z), c(X,Z))");
    for (size_t j = 0; j < r.head_args.size(); ++j)
      if (h->types[j] != T_I32) return bad(XL_UNSUPPORTED, "rule '" + r.text + "': key columns of derived relations cannot be float32");
    for (const auto* list : {&r.atoms, &r.negs})
      for (auto& a : *list) {
        Relation* rel = ctx->find(a.pred);
        if (!rel) return bad(XL_INVALID_ARGUMENT, "relation '" + a.pred + "' is not declared");
        if ((int)a.args.size() != rel->arity)
          return bad(XL_INVALID_ARGUMENT, "rule '" + r.text + "': " + a.pred + " used with " + std::to_string(a.args.size()) + " arguments but has arity " + std::to_string(rel->arity));
      }
    if (r.atoms.empty()) return bad(XL_UNSUPPORTED, "rule '" + r.text + "': a rule needs at least one body atom");
    bool found = false;
    for (auto& hi : prog->heads)
      if (hi.rel == h) {
        found = true;
        if (hi.agg != r.agg) return bad(XL_UNSUPPORTED, "relation " + h->name + " is derived with two different aggregates");
      }
    if (!found) prog->heads.push_back({h, r.agg});
  }
  // dependency graph between derived relations and Tarjan's SCC algorithm
  const int nh = (int)prog->heads.size();
  auto hid = [&](Relation* r) {
    for (int k = 0; k < nh; ++k)
      if (prog->heads[k].rel == r) return k;
    return -1;
  };
  std::vector<std::set<int>> deps(nh);
  std::vector<std::pair<int, int>> negdeps;  // (head, relation under 'not')
  for (auto& r : prog->rules) {
    for (auto& a : r.atoms) {
      int d = hid(ctx->find(a.pred));
      if (d >= 0) deps[hid(ctx->find(r.head))].insert(d);
    }
    for (auto& a : r.negs) {
      int d = hid(ctx->find(a.pred));
      if (d >= 0) {
        deps[hid(ctx->find(r.head))].insert(d);
        negdeps.push_back({hid(ctx->find(r.head)), d});
      }
    }
  }
  std::vector<int> index(nh, -1), low(nh, 0), stack;
  std::vector<bool> on(nh, false);
  std::vector<std::vector<int>> comps;
  int counter = 0;
  std::function<void(int)> visit = [&](int v) {
    index[v] = low[v] = counter++;
    stack.push_back(v);
    on[v] = true;
    for (int w : deps[v]) {
      if (index[w] < 0) {
        visit(w);
        low[v] = std::min(low[v], low[w]);
      } else if (on[w]) {
        low[v] = std::min(low[v], index[w]);
      }
    }
    if (low[v] == index[v]) {
      std::vector<int> c;
      while (true) {
        int w = stack.back();
        stack.pop_back();
        on[w] = false;
        c.push_back(w);
        if (w == v) break;
      }
      comps.push_back(c);
    }
  };
  for (int v = 0; v < nh; ++v)
    if (index[v] < 0) visit(v);
  // negation is stratified: the negated relation must be complete, i.e. in an
  // earlier component than the rule's head (Sec. 2: negative dependency edges)
  {
    std::vector<int> comp_of(nh, -1);
    for (size_t k = 0; k < comps.size(); ++k)
      for (int v : comps[k]) comp_of[v] = (int)k;
    for (auto& nd : negdeps)
      if (comp_of[nd.first] == comp_of[nd.second])
        return bad(XL_UNSUPPORTED, "relation " + prog->heads[nd.first].rel->name + " depends negatively on " +
                                       prog->heads[nd.second].rel->name + " inside one recursive component "
                                       "(negation must be stratified)");
  }
  // Tarjan emits components after everything they depend on.
  Planner pl{ctx};
  for (auto& c : comps) {
    Stratum st;
    std::set<Relation*> in;
    for (int v : c) {
      st.heads.push_back(prog->heads[v].rel);
      in.insert(prog->heads[v].rel);
    }
    st.recursive = c.size() > 1 || deps[c[0]].count(c[0]);
    // a three-column head: derived by exactly one triangle rule, outside recursion
    {
      int n3 = 0, nrules = 0, ntri = 0;
      for (int v : c) n3 += prog->heads[v].rel->arity == 3 && prog->heads[v].agg == Agg::NONE;
      for (const RuleAst& r : prog->rules)
        if (in.count(ctx->find(r.head))) {
          ++nrules;
          RulePlan tp;
          if (triangle_plan(ctx, r, &tp)) ++ntri;
        }
      if (ntri > 0 || n3 > 0) {
        if (st.recursive || c.size() != 1 || nrules != 1 || ntri != 1)
          return bad(XL_UNSUPPORTED, "a three-column relation (" + prog->heads[c[0]].rel->name +
                                         ") must be derived by one non-recursive triangle join rule alone");
        for (int ri = 0; ri < (int)prog->rules.size(); ++ri)
          if (in.count(ctx->find(prog->rules[ri].head))) {
            RulePlan tp;
            triangle_plan(ctx, prog->rules[ri], &tp);
            tp.rule = ri;
            st.full.push_back(tp);
          }
        prog->strata.push_back(st);
        continue;
      }
    }
    bool has_agg = false;
    for (int v : c) has_agg = has_agg || prog->heads[v].agg != Agg::NONE;
    if (st.recursive && has_agg) {
      if (c.size() > 1)
        return bad(XL_UNSUPPORTED, "aggregate relation " + prog->heads[c[0]].rel->name + " is mutually recursive with another relation");
      if (prog->heads[c[0]].agg == Agg::COUNT)
        return bad(XL_UNSUPPORTED, "count inside recursion is not supported (relation " + prog->heads[c[0]].rel->name + ")");
    }
    for (int ri = 0; ri < (int)prog->rules.size(); ++ri) {
      const RuleAst& r = prog->rules[ri];
      if (!in.count(ctx->find(r.head))) continue;
      std::vector<int> rec;
      for (int k = 0; k < (int)r.atoms.size(); ++k)
        if (in.count(ctx->find(r.atoms[k].pred))) rec.push_back(k);
      // Several recursive atoms (a self-join): one delta variant per
      // recursive atom, the other atoms reading the full relations
      // (Alg. 1).  Folds that are not idempotent would count a derivation
      // once per variant, so sum/logsumexp stay linear.
      if (rec.size() > 1) {
        const Agg ha = prog->head_agg(ctx->find(r.head));
        if (ha == Agg::SUM || ha == Agg::LSE)
          return bad(XL_UNSUPPORTED, "rule '" + r.text + "': sum and logsumexp need linear recursion (one recursive atom)");
      }
      // A recursive aggregate rule must carry each recursive atom's value
      // through a semiring product, so that folding each pass's
      // contributions into the relation gives the naive fixpoint's values:
      // for sum the head's value is that value itself (path sums); for
      // logsumexp that value plus other terms (a product in the log domain);
      // for min and max each recursive atom's value at most once, added
      // (a tropical product; min and max are idempotent, so passes that
      // re-derive a key change nothing).  A term added to a sum, a value that
      // enters with a minus sign, or a comparison or negated literal on a
      // carried value would act once per pass in which a key's value changes
      // instead of on the fixpoint's value.
      {
        const Agg ha = prog->head_agg(ctx->find(r.head));
        if (!rec.empty() && ha != Agg::NONE && ha != Agg::COUNT) {
          const char* an = ha == Agg::SUM ? "sum" : ha == Agg::LSE ? "logsumexp" : ha == Agg::MIN ? "min" : "max";
          const std::string why = "rule '" + r.text + "': a recursive " + an + " must carry the recursive atom's value ";
          const char* form = ha == Agg::SUM ? "unchanged (C is C1)"
                             : ha == Agg::LSE ? "plus other terms (P is P1 + ...)"
                                              : "at most once, added (D is D1 + ...)";
          for (int k : rec) {
            const Term& vt = r.atoms[k].args.back();
            if (vt.kind != Term::VAR) {
              if (ha == Agg::SUM || ha == Agg::LSE) return bad(XL_UNSUPPORTED, why + "(its value column holds no variable)");
              continue;
            }
            int uses = r.agg_var == vt.name ? 1 : 0, plus = uses;
            size_t nparts = 1;
            for (const auto& as : r.assigns) {
              int u = 0, pl = 0;
              for (const auto& pt : as.parts)
                if (pt.second.kind == Term::VAR && pt.second.name == vt.name) {
                  ++u;
                  pl += pt.first > 0;
                }
              if (as.var == r.agg_var) {
                uses += u;
                plus += pl;
                nparts = as.parts.size();
              } else if (u) {
                return bad(XL_UNSUPPORTED, why + form);  // it feeds another variable
              }
            }
            bool ok = uses == plus && uses <= 1;
            if (ha == Agg::SUM) ok = ok && uses == 1 && nparts == 1;
            if (ha == Agg::LSE) ok = ok && uses == 1;
            if (!ok) return bad(XL_UNSUPPORTED, why + form);
            for (const auto& cmp : r.cmps)
              if ((cmp.lhs.kind == Term::VAR && cmp.lhs.name == vt.name) ||
                  (cmp.rhs.kind == Term::VAR && cmp.rhs.name == vt.name))
                return bad(XL_UNSUPPORTED, why + "without comparing it");
            for (const auto& ng : r.negs)
              for (const auto& t : ng.args)
                if (t.kind == Term::VAR && t.name == vt.name)
                  return bad(XL_UNSUPPORTED, why + "without testing it in a negated literal");
          }
        }
      }
      RulePlan full;
      if (!pl.plan(r, ri, rec.empty() ? 0 : rec[0], false, &full)) return bad(pl.status, pl.err);
      st.full.push_back(full);
      for (int k : rec) {
        RulePlan var;
        if (!pl.plan(r, ri, k, true, &var)) return bad(pl.status, pl.err);
        st.variants.push_back(var);
      }
    }
    prog->strata.push_back(st);
  }
  *out = prog;
  return XL_OK;
}

std::string explain_program(const Program* p) {
  std::ostringstream os;
  auto acts = [&](const ColAct* a, int n) {
    std::ostringstream o;
    for (int j = 0; j < n; ++j) {
      if (j) o << ",";
      switch (a[j].kind) {
        case CA_BIND: o << "v" << (int)a[j].slot; break;
        case CA_CHECK_SLOT: o << "=v" << (int)a[j].slot; break;
        case CA_CHECK_CONST: o << "=#" << a[j].cval; break;
        default: o << "_";
      }
    }
    return o.str();
  };
  for (size_t s = 0; s < p->strata.size(); ++s) {
    const Stratum& st = p->strata[s];
    os << "stratum " << s << (st.recursive ? " recursive" : " non-recursive") << " heads:";
    for (Relation* h : st.heads) os << " " << h->name << "[" << agg_name(p->head_agg(h)) << "]";
    os << "\n";
    for (int pass = 0; pass < 2; ++pass) {
      const auto& plans = pass == 0 ? st.full : st.variants;
      for (const RulePlan& rp : plans) {
        os << "  " << (pass == 0 ? (st.recursive ? "seed " : "eval ") : "delta ") << "rule " << rp.rule << ": ";
        if (rp.wcoj) {
          os << "triangle join " << rp.driver->name << "(X=col " << rp.tri_a[0] << ", Y=col " << rp.tri_a[1] << ") x "
             << rp.tri_brel->name << "(Y=col " << rp.tri_b[0] << ", Z=col " << rp.tri_b[1] << ") x "
             << rp.tri_crel->name << "(X=col " << rp.tri_c[0] << ", Z=col " << rp.tri_c[1] << ") -> "
             << rp.head->name << "(X,Y,Z)\n";
          continue;
        }
        os << (rp.driver_delta ? "delta " : "scan ") << rp.driver->name << "(" << acts(rp.driver_act, rp.driver->arity) << ")";
        for (size_t k = 0; k < rp.steps.size(); ++k) {
          const StepPlan& sp = rp.steps[k];
          os << " -> join " << sp.rel->name << " on col " << sp.key_col << "=v" << sp.key_slot << " ("
             << acts(sp.act, sp.rel->arity) << ")";
        }
        for (const NegPlan& np : rp.negs) {
          os << " -> not " << np.rel->name << "(cols";
          for (int q = 0; q < np.ncols; ++q) os << " " << np.col[q];
          os << ")";
        }
        int nops = 0;
        for (auto& v : rp.stage_ops) nops += (int)v.size();
        os << " ops=" << nops << " -> " << rp.head->name << " key(v" << rp.key_slot[0];
        if (rp.nkey == 2) os << ",v" << rp.key_slot[1];
        os << ")";
        if (rp.val_slot >= 0) os << " val v" << rp.val_slot;
        if (rp.carried) os << " [grouped by v" << rp.key_slot[0] << "]";
        if (rp.carried_val) os << " [keyed by v" << rp.key_slot[0] << ", v" << rp.key_slot[1] << "]";
        GatherShape gs;
        if (gather_shape(rp, &gs)) os << " [gathered by head row v" << rp.key_slot[0] << "]";
        os << "\n";
      }
    }
  }
  return os.str();
}

}  // namespace xlh
