// qasm.cpp -- OpenQASM front end of the compile phase (Sec. 3: a normalized
// OpenQASM circuit is lowered once into an internal gate sequence; Algorithm 1,
// compile phase: parse C into G = {(g_i, w_i, p_i)}).
//
// Accepted: OpenQASM 2.0 and the static subset of OpenQASM 3 --
//   OPENQASM v; include "qelib1.inc" | "stdgates.inc";
//   qreg r[n]; | qubit[n] r; | qubit r;      (registers flattened in order)
//   creg c[n]; | bit[n] c; | bit c;          (ignored)
//   input float[..] name; | input angle name; | input array[float[..], n] name;
//   gate name(a, b) q0, q1 { ... }           (expanded at each call)
//   barrier ...; | gphase(x);                (no effect on the outputs)
//   measure q -> c; | c = measure q;         (terminal: no later gate may
//                                             touch a measured qubit)
//   gate calls with register broadcasting, the standard gate library.
// Angles are expressions over numbers, pi / tau / euler, the declared inputs
// (scalars or array elements), + - * / ^ and sin cos tan exp ln sqrt; the
// result must be a constant or affine in one input (mul * value + add).
// Declared inputs named in `input_names` are data features (inputs[b, .]);
// every other declared input is a trainable parameter.  Slots are assigned
// in declaration order, an array taking consecutive slots.
// Rejected with the construct named: reset, mid-circuit measurement, classical
// control, loops, subroutines, gate modifiers, opaque gates, other includes.
//
// Host-only code: no device calls.
#include <algorithm>
#include <cctype>
#include <cmath>
#include <cstring>
#include <map>
#include <memory>
#include <set>
#include <string>
#include <vector>

#include "vqc.h"

namespace {

constexpr double kPi = 3.14159265358979323846;

struct Tok {
  enum Kind { END, ID, NUM, STR, SYM } kind = END;
  std::string text;
  double num = 0.0;
  int line = 0, col = 0;
};

struct Error {
  int code;
  std::string msg;
};

std::vector<Tok> lex(const std::string& s) {
  std::vector<Tok> out;
  size_t i = 0;
  int line = 1, col = 1;
  auto adv = [&](size_t k) {
    for (size_t j = 0; j < k && i < s.size(); ++j, ++i) {
      if (s[i] == '\n') {
        ++line;
        col = 1;
      } else {
        ++col;
      }
    }
  };
  while (i < s.size()) {
    const char c = s[i];
    if (std::isspace((unsigned char)c)) {
      adv(1);
      continue;
    }
    if (c == '/' && i + 1 < s.size() && s[i + 1] == '/') {
      while (i < s.size() && s[i] != '\n') adv(1);
      continue;
    }
    if (c == '/' && i + 1 < s.size() && s[i + 1] == '*') {
      adv(2);
      while (i < s.size() && !(s[i] == '*' && i + 1 < s.size() && s[i + 1] == '/')) adv(1);
      if (i >= s.size()) throw Error{VQC_ERR_INVALID_ARG, "unterminated comment"};
      adv(2);
      continue;
    }
    Tok t;
    t.line = line;
    t.col = col;
    // the UTF-8 letters OpenQASM 3 uses for its constants
    if (s.compare(i, 2, "\xcf\x80") == 0 || s.compare(i, 2, "\xcf\x84") == 0 ||
        s.compare(i, 3, "\xe2\x84\x87") == 0) {
      const bool three = s.compare(i, 3, "\xe2\x84\x87") == 0;
      t.kind = Tok::ID;
      t.text = s.compare(i, 2, "\xcf\x80") == 0 ? "pi" : s.compare(i, 2, "\xcf\x84") == 0 ? "tau"
                                                                                         : "euler";
      i += three ? 3 : 2;
      col += 1;
      out.push_back(t);
      continue;
    }
    if (std::isalpha((unsigned char)c) || c == '_') {
      size_t j = i;
      while (j < s.size() && (std::isalnum((unsigned char)s[j]) || s[j] == '_')) ++j;
      t.kind = Tok::ID;
      t.text = s.substr(i, j - i);
      adv(j - i);
      out.push_back(t);
      continue;
    }
    if (std::isdigit((unsigned char)c) || (c == '.' && i + 1 < s.size() &&
                                           std::isdigit((unsigned char)s[i + 1]))) {
      const char* begin = s.c_str() + i;
      char* end = nullptr;
      t.num = std::strtod(begin, &end);
      const size_t len = (size_t)(end - begin);
      t.kind = Tok::NUM;
      t.text = s.substr(i, len);
      adv(len);
      out.push_back(t);
      continue;
    }
    if (c == '"') {
      size_t j = i + 1;
      while (j < s.size() && s[j] != '"' && s[j] != '\n') ++j;
      if (j >= s.size() || s[j] != '"')
        throw Error{VQC_ERR_INVALID_ARG, "line " + std::to_string(line) + ": unterminated string"};
      t.kind = Tok::STR;
      t.text = s.substr(i + 1, j - i - 1);
      adv(j + 1 - i);
      out.push_back(t);
      continue;
    }
    static const char* two[] = {"->", "**", "==", "!=", "<=", ">=", "&&", "||", "++", "+=", "-="};
    bool matched = false;
    for (const char* op : two)
      if (s.compare(i, 2, op) == 0) {
        t.kind = Tok::SYM;
        t.text = op;
        adv(2);
        out.push_back(t);
        matched = true;
        break;
      }
    if (matched) continue;
    if (std::strchr(";,()[]{}+-*/^=@<>!&|%~:.#$", c)) {
      t.kind = Tok::SYM;
      t.text = std::string(1, c);
      adv(1);
      out.push_back(t);
      continue;
    }
    throw Error{VQC_ERR_INVALID_ARG, "line " + std::to_string(line) + ":" + std::to_string(col) +
                                         ": unexpected character"};
  }
  Tok e;
  e.kind = Tok::END;
  e.line = line;
  e.col = col;
  out.push_back(e);
  return out;
}

// A real value that is constant (src < 0) or mul * value(src, idx) + add.
struct Affine {
  int src = -1, idx = 0;
  double mul = 0.0, add = 0.0;
  bool constant() const { return src < 0; }
};

struct Symbol {  // a declared input: slots [base, base + size) of params or inputs
  int src, base, size;
  bool array;
};

struct GateDef {
  std::vector<std::string> params, qargs;
  std::vector<Tok> body;  // tokens between the braces, END-terminated
};

struct Register {
  int base, size;
};

class Parser {
 public:
  Parser(const std::string& src, const std::set<std::string>& data_names)
      : data_names_(data_names) {
    toks_ = lex(src);
  }

  void run() {
    size_t pos = 0;
    Ctx top;
    top.toks = &toks_;
    top.pos = &pos;
    while (toks_[pos].kind != Tok::END) statement(top);
    for (const std::string& name : data_names_)
      if (!used_names_.count(name))
        throw Error{VQC_ERR_INVALID_ARG, "input name '" + name + "' is not declared"};
  }

  std::vector<vqc_op> ops;
  int n_qubits = 0, n_params = 0, n_inputs = 0;

 private:
  // a token stream with the substitutions of one gate expansion
  struct Ctx {
    const std::vector<Tok>* toks = nullptr;
    size_t* pos = nullptr;
    const std::map<std::string, Affine>* params = nullptr;  // gate parameters
    const std::map<std::string, int>* qargs = nullptr;      // gate qubit arguments
    int depth = 0;
    // the stream ends with an END token, which is never consumed
    const Tok& peek(int k = 0) const {
      return (*toks)[std::min(*pos + (size_t)k, toks->size() - 1)];
    }
    const Tok& next() {
      const Tok& t = (*toks)[*pos];
      if (t.kind != Tok::END) ++*pos;
      return t;
    }
  };

  [[noreturn]] void err(const Tok& t, const std::string& m, int code = VQC_ERR_INVALID_ARG) {
    throw Error{code, "line " + std::to_string(t.line) + ":" + std::to_string(t.col) + ": " + m};
  }
  [[noreturn]] void unsupported(const Tok& t, const std::string& what) {
    err(t, what + " is not supported (static circuits only)", VQC_ERR_UNSUPPORTED);
  }

  void expect(Ctx& c, const char* sym) {
    const Tok& t = c.next();
    if (t.kind != Tok::SYM || t.text != sym) err(t, std::string("expected '") + sym + "'");
  }
  bool accept(Ctx& c, const char* sym) {
    if (c.peek().kind == Tok::SYM && c.peek().text == sym) {
      ++*c.pos;
      return true;
    }
    return false;
  }
  std::string ident(Ctx& c) {
    const Tok& t = c.next();
    if (t.kind != Tok::ID) err(t, "expected a name");
    return t.text;
  }
  int integer(Ctx& c) {
    const Tok& t = c.next();
    if (t.kind != Tok::NUM || t.num != std::floor(t.num) || t.num < 0 || t.num > 1e6)
      err(t, "expected a non-negative integer");
    return (int)t.num;
  }
  void skip_statement(Ctx& c) {
    while (c.peek().kind != Tok::END && !(c.peek().kind == Tok::SYM && c.peek().text == ";"))
      ++*c.pos;
    expect(c, ";");
  }

  void declare_name(const Tok& t, const std::string& name) {
    if (registers_.count(name) || symbols_.count(name) || gates_.count(name) ||
        bit_names_.count(name))
      err(t, "'" + name + "' is already declared");
  }

  // ------------------------------------------------------------ statements
  void statement(Ctx& c) {
    const Tok& t = c.peek();
    if (t.kind != Tok::ID) err(t, "expected a statement");
    const std::string& w = t.text;
    if (w == "OPENQASM") {
      ++*c.pos;
      skip_statement(c);
    } else if (w == "include") {
      ++*c.pos;
      const Tok& f = c.next();
      if (f.kind != Tok::STR) err(f, "expected a file name");
      if (f.text != "qelib1.inc" && f.text != "stdgates.inc")
        err(f, "include of '" + f.text + "'", VQC_ERR_UNSUPPORTED);
      expect(c, ";");
    } else if (w == "qreg" || w == "creg") {
      ++*c.pos;
      const Tok& nt = c.peek();
      const std::string name = ident(c);
      expect(c, "[");
      const int n = integer(c);
      expect(c, "]");
      expect(c, ";");
      declare_name(nt, name);
      if (w == "qreg") add_register(nt, name, n);
      else bit_names_.insert(name);
    } else if (w == "qubit" || w == "bit") {
      ++*c.pos;
      int n = 1;
      if (accept(c, "[")) {
        n = integer(c);
        expect(c, "]");
      }
      const Tok& nt = c.peek();
      const std::string name = ident(c);
      if (accept(c, "=")) {  // bit c = measure q;
        if (w == "qubit") err(nt, "qubits cannot be assigned");
        bit_names_.insert(name);
        measure_rhs(c);
        return;
      }
      expect(c, ";");
      declare_name(nt, name);
      if (w == "qubit") add_register(nt, name, n);
      else bit_names_.insert(name);
    } else if (w == "input") {
      ++*c.pos;
      input_decl(c);
    } else if (w == "gate") {
      ++*c.pos;
      gate_def(c);
    } else if (w == "barrier") {
      ++*c.pos;
      skip_statement(c);
    } else if (w == "gphase") {  // a global phase: no output depends on it
      ++*c.pos;
      skip_statement(c);
    } else if (w == "measure") {
      ++*c.pos;
      measure_qubits(c);
      if (accept(c, "->")) skip_target(c);
      expect(c, ";");
    } else if (bit_names_.count(w) && (c.peek(1).text == "=" || c.peek(1).text == "[")) {
      // c = measure q;  or  c[i] = measure q[i];
      ++*c.pos;
      if (accept(c, "[")) {
        integer(c);
        expect(c, "]");
      }
      expect(c, "=");
      measure_rhs(c);
    } else if (w == "reset") {
      unsupported(t, "reset");
    } else if (w == "if" || w == "while" || w == "for" || w == "switch") {
      unsupported(t, "classical control ('" + w + "')");
    } else if (w == "def" || w == "defcal" || w == "cal" || w == "extern" || w == "box" ||
               w == "delay" || w == "return") {
      unsupported(t, "'" + w + "'");
    } else if (w == "opaque") {
      unsupported(t, "an opaque gate");
    } else if (w == "ctrl" || w == "negctrl" || w == "inv" || w == "pow") {
      unsupported(t, "the gate modifier '" + w + "'");
    } else if (w == "const" || w == "float" || w == "int" || w == "uint" || w == "angle" ||
               w == "bool" || w == "complex" || w == "let" || w == "output") {
      unsupported(t, "classical declaration '" + w + "'");
    } else {
      gate_call(c);
    }
  }

  void add_register(const Tok& t, const std::string& name, int n) {
    if (n < 1) err(t, "a register needs at least one qubit");
    if (n_qubits + n > VQC_MAX_QUBITS)
      err(t, "more than " + std::to_string(VQC_MAX_QUBITS) + " qubits", VQC_ERR_TOO_LARGE);
    registers_[name] = {n_qubits, n};
    n_qubits += n;
  }

  void input_decl(Ctx& c) {
    int size = 1;
    bool array = false;
    const Tok& ty = c.peek();
    const std::string type = ident(c);
    if (type == "array") {
      expect(c, "[");
      const std::string et = ident(c);
      if (et != "float" && et != "angle") err(ty, "input arrays must hold float or angle");
      if (accept(c, "[")) {
        integer(c);
        expect(c, "]");
      }
      expect(c, ",");
      size = integer(c);
      expect(c, "]");
      array = true;
    } else if (type == "float" || type == "angle") {
      if (accept(c, "[")) {
        integer(c);
        expect(c, "]");
      }
    } else {
      err(ty, "inputs must be float, angle or arrays of them");
    }
    const Tok& nt = c.peek();
    const std::string name = ident(c);
    expect(c, ";");
    declare_name(nt, name);
    if (size < 1) err(nt, "an input array needs at least one element");
    const bool data = data_names_.count(name) > 0;
    Symbol s;
    s.src = data ? VQC_SRC_INPUT : VQC_SRC_PARAM;
    s.base = data ? n_inputs : n_params;
    s.size = size;
    s.array = array;
    (data ? n_inputs : n_params) += size;
    symbols_[name] = s;
    used_names_.insert(name);
  }

  void gate_def(Ctx& c) {
    const Tok& nt = c.peek();
    const std::string name = ident(c);
    declare_name(nt, name);  // a definition of a standard gate's name replaces it
    auto g = std::make_unique<GateDef>();
    if (accept(c, "(")) {
      if (!accept(c, ")")) {
        do g->params.push_back(ident(c));
        while (accept(c, ","));
        expect(c, ")");
      }
    }
    do g->qargs.push_back(ident(c));
    while (accept(c, ","));
    expect(c, "{");
    int depth = 1;
    while (true) {
      const Tok& t = c.next();
      if (t.kind == Tok::END) err(t, "unterminated gate body");
      if (t.kind == Tok::SYM && t.text == "{") ++depth;
      if (t.kind == Tok::SYM && t.text == "}" && --depth == 0) break;
      g->body.push_back(t);
    }
    Tok e;
    e.kind = Tok::END;
    e.line = nt.line;
    e.col = nt.col;
    g->body.push_back(e);
    gates_[name] = std::move(g);
  }

  // ------------------------------------------------------------ measurement
  void measure_rhs(Ctx& c) {
    const Tok& t = c.next();
    if (t.kind != Tok::ID || t.text != "measure") err(t, "expected 'measure'");
    measure_qubits(c);
    expect(c, ";");
  }
  void measure_qubits(Ctx& c) {
    for (int q : qubit_operand(c)) measured_.insert(q);
  }
  void skip_target(Ctx& c) {
    ident(c);
    if (accept(c, "[")) {
      integer(c);
      expect(c, "]");
    }
  }

  // One operand: a qubit (reg[i], or a gate's qubit argument) or a whole register.
  std::vector<int> qubit_operand(Ctx& c) {
    const Tok& t = c.peek();
    const std::string name = ident(c);
    if (c.qargs) {
      auto it = c.qargs->find(name);
      if (it == c.qargs->end()) err(t, "'" + name + "' is not a qubit argument of the gate");
      return {it->second};
    }
    auto it = registers_.find(name);
    if (it == registers_.end()) err(t, "'" + name + "' is not a quantum register");
    if (accept(c, "[")) {
      const Tok& it2 = c.peek();
      const int i = integer(c);
      expect(c, "]");
      if (i >= it->second.size)
        err(it2, "index " + std::to_string(i) + " out of range for '" + name + "'");
      return {it->second.base + i};
    }
    std::vector<int> all;
    for (int i = 0; i < it->second.size; ++i) all.push_back(it->second.base + i);
    return all;
  }

  // ------------------------------------------------------------ gate calls
  struct Builtin {
    int kind, wires, angles;
  };
  static const Builtin* builtin(const std::string& name) {
    static const std::map<std::string, Builtin> table = {
        {"id", {VQC_ID, 1, 0}},     {"x", {VQC_X, 1, 0}},        {"y", {VQC_Y, 1, 0}},
        {"z", {VQC_Z, 1, 0}},       {"h", {VQC_H, 1, 0}},        {"s", {VQC_S, 1, 0}},
        {"sdg", {VQC_SDG, 1, 0}},   {"t", {VQC_T, 1, 0}},        {"tdg", {VQC_TDG, 1, 0}},
        {"sx", {VQC_SX, 1, 0}},     {"sxdg", {VQC_SXDG, 1, 0}},  {"rx", {VQC_RX, 1, 1}},
        {"ry", {VQC_RY, 1, 1}},     {"rz", {VQC_RZ, 1, 1}},      {"p", {VQC_P, 1, 1}},
        {"u1", {VQC_P, 1, 1}},      {"phase", {VQC_P, 1, 1}},    {"u2", {VQC_U2, 1, 2}},
        {"u3", {VQC_U3, 1, 3}},     {"u", {VQC_U3, 1, 3}},       {"U", {VQC_U3, 1, 3}},
        {"cx", {VQC_CNOT, 2, 0}},   {"CX", {VQC_CNOT, 2, 0}},    {"cnot", {VQC_CNOT, 2, 0}},
        {"cy", {VQC_CY, 2, 0}},     {"cz", {VQC_CZ, 2, 0}},      {"ch", {VQC_CH, 2, 0}},
        {"swap", {VQC_SWAP, 2, 0}}, {"crx", {VQC_CRX, 2, 1}},    {"cry", {VQC_CRY, 2, 1}},
        {"crz", {VQC_CRZ, 2, 1}},   {"cp", {VQC_CP, 2, 1}},      {"cu1", {VQC_CP, 2, 1}},
        {"cphase", {VQC_CP, 2, 1}}, {"rxx", {VQC_RXX, 2, 1}},    {"ryy", {VQC_RYY, 2, 1}},
        {"rzz", {VQC_RZZ, 2, 1}},   {"ccx", {VQC_CCX, 3, 0}},    {"toffoli", {VQC_CCX, 3, 0}},
        {"cswap", {VQC_CSWAP, 3, 0}}, {"fredkin", {VQC_CSWAP, 3, 0}},
    };
    auto it = table.find(name);
    return it == table.end() ? nullptr : &it->second;
  }

  void gate_call(Ctx& c) {
    const Tok& nt = c.peek();
    const std::string name = ident(c);
    auto gi = gates_.find(name);
    const Builtin* b = gi == gates_.end() ? builtin(name) : nullptr;
    if (!b && gi == gates_.end()) {
      if (name == "measure" || name == "reset") unsupported(nt, name);
      err(nt, "unknown gate '" + name + "'", VQC_ERR_UNSUPPORTED);
    }
    std::vector<Affine> args;
    if (accept(c, "(")) {
      if (!accept(c, ")")) {
        do args.push_back(expr(c));
        while (accept(c, ","));
        expect(c, ")");
      }
    }
    std::vector<std::vector<int>> operands;
    do operands.push_back(qubit_operand(c));
    while (accept(c, ","));
    expect(c, ";");
    const int want_args = b ? b->angles : (int)gi->second->params.size();
    const int want_qubits = b ? b->wires : (int)gi->second->qargs.size();
    if ((int)args.size() != want_args)
      err(nt, "'" + name + "' takes " + std::to_string(want_args) + " angle(s), got " +
                  std::to_string(args.size()));
    if ((int)operands.size() != want_qubits)
      err(nt, "'" + name + "' acts on " + std::to_string(want_qubits) + " qubit(s), got " +
                  std::to_string(operands.size()));
    // register broadcasting: whole registers of one size, single qubits repeated
    size_t reps = 1;
    for (const auto& o : operands)
      if (o.size() > 1) {
        if (reps > 1 && o.size() != reps) err(nt, "registers of different sizes in one call");
        reps = o.size();
      }
    for (size_t r = 0; r < reps; ++r) {
      std::vector<int> qs;
      for (const auto& o : operands) qs.push_back(o.size() > 1 ? o[r] : o[0]);
      for (size_t i = 0; i < qs.size(); ++i)
        for (size_t j = 0; j < i; ++j)
          if (qs[i] == qs[j]) err(nt, "'" + name + "' uses a qubit twice");
      for (int q : qs)
        if (measured_.count(q))
          unsupported(nt, "a gate after measuring its qubit (mid-circuit measurement)");
      if (b) emit(nt, *b, args, qs);
      else expand(nt, *gi->second, args, qs, c.depth);
    }
  }

  void emit(const Tok& t, const Builtin& b, const std::vector<Affine>& args,
            const std::vector<int>& qs) {
    vqc_op op;
    std::memset(&op, 0, sizeof(op));
    op.kind = b.kind;
    for (int i = 0; i < 3; ++i) op.wires[i] = i < (int)qs.size() ? qs[i] : -1;
    for (int s = 0; s < b.angles; ++s) {
      const Affine& a = args[s];
      if (!std::isfinite(a.add) || !std::isfinite(a.mul)) err(t, "angle is not finite");
      if (a.constant()) {
        op.src[s] = VQC_SRC_CONST;
        op.val[s] = (float)a.add;
        op.mul[s] = 1.f;
      } else {
        op.src[s] = a.src;
        op.idx[s] = a.idx;
        op.mul[s] = (float)a.mul;
        op.val[s] = (float)a.add;
      }
    }
    if (ops.size() >= (size_t)(1 << 20)) err(t, "more than 2^20 gates", VQC_ERR_TOO_LARGE);
    ops.push_back(op);
  }

  void expand(const Tok& t, const GateDef& g, const std::vector<Affine>& args,
              const std::vector<int>& qs, int depth) {
    if (depth > 64) err(t, "gate definitions nest more than 64 deep", VQC_ERR_TOO_LARGE);
    std::map<std::string, Affine> pm;
    for (size_t i = 0; i < g.params.size(); ++i) pm[g.params[i]] = args[i];
    std::map<std::string, int> qm;
    for (size_t i = 0; i < g.qargs.size(); ++i) qm[g.qargs[i]] = qs[i];
    size_t pos = 0;
    Ctx c;
    c.toks = &g.body;
    c.pos = &pos;
    c.params = &pm;
    c.qargs = &qm;
    c.depth = depth + 1;
    while (c.peek().kind != Tok::END) {
      const Tok& s = c.peek();
      if (s.kind == Tok::ID && s.text == "barrier") {
        ++pos;
        skip_statement(c);
      } else if (s.kind == Tok::ID && s.text == "gphase") {
        ++pos;
        skip_statement(c);
      } else if (s.kind == Tok::ID && (s.text == "ctrl" || s.text == "inv" || s.text == "pow" ||
                                       s.text == "negctrl")) {
        unsupported(s, "the gate modifier '" + s.text + "'");
      } else {
        gate_call(c);
      }
    }
  }

  // ------------------------------------------------------------ expressions
  Affine konst(double v) {
    Affine a;
    a.add = v;
    return a;
  }

  // Angle expressions nest at most kMaxNest deep (parentheses, signs, powers,
  // function calls): the parser recurses once per level.
  static constexpr int kMaxNest = 256;
  int nest_ = 0;
  struct Nest {
    int& d;
    Nest(Parser* p, const Tok& t) : d(p->nest_) {
      if (d >= kMaxNest) p->err(t, "angle expression nests more than 256 deep", VQC_ERR_TOO_LARGE);
      ++d;
    }
    ~Nest() { --d; }
  };

  Affine expr(Ctx& c) {
    Nest guard(this, c.peek());
    Affine a = term(c);
    while (c.peek().kind == Tok::SYM && (c.peek().text == "+" || c.peek().text == "-")) {
      const Tok& op = c.next();
      Affine b = term(c);
      a = add(op, a, b, op.text == "-" ? -1.0 : 1.0);
    }
    return a;
  }
  Affine term(Ctx& c) {
    Affine a = unary(c);
    while (c.peek().kind == Tok::SYM && (c.peek().text == "*" || c.peek().text == "/")) {
      const Tok& op = c.next();
      Affine b = unary(c);
      if (op.text == "*") {
        if (a.constant()) a = scale(b, a.add);
        else if (b.constant()) a = scale(a, b.add);
        else err(op, "angle is not affine in one input (product of inputs)");
      } else {
        if (!b.constant()) err(op, "angle is not affine in one input (division by an input)");
        if (b.add == 0.0) err(op, "division by zero");
        a = scale(a, 1.0 / b.add);
      }
    }
    return a;
  }
  Affine unary(Ctx& c) {
    Nest guard(this, c.peek());
    if (accept(c, "-")) return scale(unary(c), -1.0);
    if (accept(c, "+")) return unary(c);
    return power(c);
  }
  Affine power(Ctx& c) {
    Affine a = primary(c);
    if (c.peek().kind == Tok::SYM && (c.peek().text == "^" || c.peek().text == "**")) {
      const Tok& op = c.next();
      Affine b = unary(c);
      if (!a.constant() || !b.constant()) err(op, "angle is not affine in one input (power)");
      return konst(std::pow(a.add, b.add));
    }
    return a;
  }
  Affine primary(Ctx& c) {
    const Tok& t = c.next();
    if (t.kind == Tok::NUM) return konst(t.num);
    if (t.kind == Tok::SYM && t.text == "(") {
      Affine a = expr(c);
      expect(c, ")");
      return a;
    }
    if (t.kind != Tok::ID) err(t, "expected an angle expression");
    const std::string& w = t.text;
    if (c.params) {
      auto it = c.params->find(w);
      if (it != c.params->end()) return it->second;
    }
    if (w == "pi") return konst(kPi);
    if (w == "tau") return konst(2 * kPi);
    if (w == "euler") return konst(std::exp(1.0));
    static const std::map<std::string, double (*)(double)> fns = {
        {"sin", [](double v) { return std::sin(v); }},  {"cos", [](double v) { return std::cos(v); }},
        {"tan", [](double v) { return std::tan(v); }},  {"exp", [](double v) { return std::exp(v); }},
        {"ln", [](double v) { return std::log(v); }},   {"sqrt", [](double v) { return std::sqrt(v); }},
        {"arcsin", [](double v) { return std::asin(v); }},
        {"arccos", [](double v) { return std::acos(v); }},
        {"arctan", [](double v) { return std::atan(v); }}};
    auto f = fns.find(w);
    if (f != fns.end()) {
      expect(c, "(");
      Affine a = expr(c);
      expect(c, ")");
      if (!a.constant()) err(t, "angle is not affine in one input (" + w + " of an input)");
      return konst(f->second(a.add));
    }
    auto s = symbols_.find(w);
    if (s == symbols_.end()) err(t, "unknown name '" + w + "' in an angle");
    int i = 0;
    if (s->second.array) {
      expect(c, "[");
      const Tok& it = c.peek();
      i = integer(c);
      expect(c, "]");
      if (i >= s->second.size) err(it, "index " + std::to_string(i) + " out of range for '" + w + "'");
    }
    Affine a;
    a.src = s->second.src;
    a.idx = s->second.base + i;
    a.mul = 1.0;
    return a;
  }
  Affine scale(Affine a, double k) {
    a.add *= k;
    if (!a.constant()) a.mul *= k;
    if (!a.constant() && a.mul == 0.0) return konst(a.add);
    return a;
  }
  Affine add(const Tok& op, Affine a, Affine b, double sign) {
    b = scale(b, sign);
    if (a.constant()) {
      b.add += a.add;
      return b;
    }
    if (b.constant()) {
      a.add += b.add;
      return a;
    }
    if (a.src != b.src || a.idx != b.idx)
      err(op, "angle is not affine in one input (two different inputs)");
    a.mul += b.mul;
    a.add += b.add;
    if (a.mul == 0.0) return konst(a.add);
    return a;
  }

  std::vector<Tok> toks_;
  std::set<std::string> data_names_, used_names_, bit_names_;
  std::map<std::string, Register> registers_;
  std::map<std::string, Symbol> symbols_;
  std::map<std::string, std::unique_ptr<GateDef>> gates_;
  std::set<int> measured_;
};

std::set<std::string> split_names(const char* names) {
  std::set<std::string> out;
  if (!names) return out;
  std::string cur;
  for (const char* p = names;; ++p) {
    if (*p == ',' || *p == '\0') {
      size_t a = 0, b = cur.size();
      while (a < b && std::isspace((unsigned char)cur[a])) ++a;
      while (b > a && std::isspace((unsigned char)cur[b - 1])) --b;
      if (b > a) out.insert(cur.substr(a, b - a));
      cur.clear();
      if (*p == '\0') break;
    } else {
      cur += *p;
    }
  }
  return out;
}

}  // namespace

namespace vqc {

int parse_qasm(const char* source, const char* input_names, std::vector<vqc_op>& ops,
               int& n_qubits, int& n_params, int& n_inputs, std::string& msg) {
  if (!source) {
    msg = "source is NULL";
    return VQC_ERR_INVALID_ARG;
  }
  try {
    Parser p(source, split_names(input_names));
    p.run();
    if (p.n_qubits == 0) {
      msg = "the program declares no qubits";
      return VQC_ERR_INVALID_ARG;
    }
    ops = std::move(p.ops);
    n_qubits = p.n_qubits;
    n_params = p.n_params;
    n_inputs = p.n_inputs;
    return VQC_OK;
  } catch (const Error& e) {
    msg = e.msg;
    return e.code;
  } catch (const std::bad_alloc&) {
    msg = "out of host memory";
    return VQC_ERR_OOM;
  }
}

}  // namespace vqc
