// libpartir planner: PartIR:Core value tiling and propagation on the host.
//
// A schedule of ManualPartition tactics (Sec. 3) is desugared into compiler
// actions -- value tiling `tile<%v, dim, axis>` followed by `propagate` --
// and applied to a small tensor program (matmul / add / gelu / rmsnorm on
// 2-D values).  Propagation (Sec. 5.2.2) wraps operations in loops using the
// tile-mapping registry (TMR, Sec. 5.2.1):
//   * forward: an entry whose tiled operands are all available tiled on the
//     axis (produced by a #tile loop or by value tiling);
//   * backward: an entry whose result action is #tile<d> when the result is
//     used sliced along d downstream;
//   * inference (partial match): when no entry matches fully and exactly one
//     entry matches some operands while its other operands are untiled on
//     the axis, those operands are sliced as the entry asks.
// Several candidates make a conflict, which is reported and left alone
// (Sec. 5.2.3); an operation already inside a loop over an axis never gets a
// second loop over it.  Every axis keeps its own state, so multi-axis nests
// and deep tiling (App. A) compose: the loop order of an operation is the
// order in which its loops were introduced.
//
// The planner then names the libpartir entry point that executes each loop
// nest it recognises (a single partitioned matmul, the Megatron MLP block).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "../../include/partir.h"

namespace partir {
namespace planner {

constexpr int NONE = -1;   // operand not sliced / value not tiled / no loop on the axis
constexpr int SUM = -2;    // the #sum loop action

// A TMR entry: per-operand tiling dim (or NONE) and the loop action it yields.
struct Entry {
  std::vector<int> in;
  int out;
};

const std::vector<Entry>& tmr(const std::string& kind) {
  // matmul: (#tile<0>, _) -> #tile<0>; (_, #tile<1>) -> #tile<1>; (#tile<1>, #tile<0>) -> #sum
  static const std::vector<Entry> matmul = {{{0, NONE}, 0}, {{NONE, 1}, 1}, {{1, 0}, SUM}};
  // element-wise binary op: both operands tiled alike, result tiled the same way
  static const std::vector<Entry> binary = {{{0, 0}, 0}, {{1, 1}, 1}};
  static const std::vector<Entry> unary = {{{0}, 0}, {{1}, 1}};
  // rmsnorm reduces over dim 1: only its rows are independent
  static const std::vector<Entry> rowwise = {{{0}, 0}};
  static const std::vector<Entry> none;
  if (kind == "matmul") return matmul;
  if (kind == "add") return binary;
  if (kind == "gelu") return unary;
  if (kind == "rmsnorm") return rowwise;
  return none;
}

int arity(const std::string& kind) {
  if (kind == "matmul" || kind == "add") return 2;
  if (kind == "gelu" || kind == "rmsnorm") return 1;
  return -1;
}

struct Value {
  std::string name;
  int64_t dim[2];
  int producer = -1;   // op index, -1 for a function argument
};

struct Op {
  std::string kind;
  std::vector<int> in;
  int out;
};

struct Axis {
  std::string name;
  int size;
};

struct Error {
  int status;
  std::string msg;
};

Error err(int status, const char* fmt, ...) {
  char buf[400];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return Error{status, buf};
}

std::vector<std::string> split_ws(const std::string& line) {
  std::istringstream is(line);
  std::vector<std::string> t;
  std::string w;
  while (is >> w) t.push_back(w);
  return t;
}

std::vector<std::string> lines_of(const char* text) {
  std::vector<std::string> out;
  std::string cur;
  for (const char* c = text; *c; ++c) {
    if (*c == '\n' || *c == ';') {
      out.push_back(cur);
      cur.clear();
    } else {
      cur.push_back(*c);
    }
  }
  out.push_back(cur);
  for (auto& l : out) {
    const size_t h = l.find('#');
    if (h != std::string::npos) l.resize(h);
  }
  return out;
}

bool parse_int(const std::string& s, int64_t& v) {
  if (s.empty()) return false;
  char* end = nullptr;
  v = strtoll(s.c_str(), &end, 10);
  return end && *end == 0;
}

class Planner {
 public:
  std::vector<Axis> axes;
  std::vector<Value> values;
  std::vector<Op> ops;
  std::map<std::string, int> by_name;
  std::vector<int> rets;

  // per-axis state
  std::vector<std::vector<int>> vtile;                 // [value][axis]: dim available tiled, or NONE
  std::vector<std::vector<int>> vslice;                // [value][axis]: dim it was value-tiled along (a sliced use)
  std::vector<std::vector<int>> loop;                  // [op][axis]: NONE, tile dim or SUM
  std::vector<std::vector<int>> order;                 // [op]: axes, outer first
  std::vector<std::vector<std::vector<int>>> slice;    // [op][operand][axis]: dim or NONE
  std::set<std::pair<int, int>> conflicts;             // (op, axis)
  std::vector<std::string> actions;

  int axis_index(const std::string& n) const {
    for (size_t i = 0; i < axes.size(); ++i)
      if (axes[i].name == n) return (int)i;
    return -1;
  }

  Error parse_program(const char* text) {
    const auto ls = lines_of(text);
    for (size_t ln = 0; ln < ls.size(); ++ln) {
      const auto t = split_ws(ls[ln]);
      if (t.empty()) continue;
      if (t[0] == "mesh") {
        for (size_t i = 1; i < t.size(); ++i) {
          const size_t eq = t[i].find('=');
          int64_t sz;
          if (eq == std::string::npos || !parse_int(t[i].substr(eq + 1), sz) || sz < 1)
            return err(PARTIR_E_SHAPE, "line %zu: mesh axis '%s' must be name=size", ln + 1, t[i].c_str());
          if (axis_index(t[i].substr(0, eq)) >= 0)
            return err(PARTIR_E_AXIS, "line %zu: axis '%s' declared twice", ln + 1, t[i].substr(0, eq).c_str());
          axes.push_back(Axis{t[i].substr(0, eq), (int)sz});
        }
      } else if (t[0] == "arg") {
        if (t.size() != 3) return err(PARTIR_E_SHAPE, "line %zu: arg <name> <rows>x<cols>", ln + 1);
        const size_t x = t[2].find('x');
        int64_t r, c;
        if (x == std::string::npos || !parse_int(t[2].substr(0, x), r) || !parse_int(t[2].substr(x + 1), c) || r < 0 || c < 0)
          return err(PARTIR_E_SHAPE, "line %zu: bad shape '%s'", ln + 1, t[2].c_str());
        if (by_name.count(t[1])) return err(PARTIR_E_SHAPE, "line %zu: '%s' defined twice", ln + 1, t[1].c_str());
        by_name[t[1]] = (int)values.size();
        values.push_back(Value{t[1], {r, c}, -1});
      } else if (t[0] == "ret") {
        for (size_t i = 1; i < t.size(); ++i) {
          if (!by_name.count(t[i])) return err(PARTIR_E_SHAPE, "line %zu: unknown value '%s'", ln + 1, t[i].c_str());
          rets.push_back(by_name[t[i]]);
        }
      } else if (t.size() >= 3 && t[1] == "=") {
        const std::string kind = t[2];
        const int n = arity(kind);
        if (n < 0) return err(PARTIR_E_UNSUPPORTED, "line %zu: unknown op '%s'", ln + 1, kind.c_str());
        if ((int)t.size() != 3 + n) return err(PARTIR_E_SHAPE, "line %zu: %s takes %d operands", ln + 1, kind.c_str(), n);
        if (by_name.count(t[0])) return err(PARTIR_E_SHAPE, "line %zu: '%s' defined twice", ln + 1, t[0].c_str());
        Op op;
        op.kind = kind;
        for (int i = 0; i < n; ++i) {
          if (!by_name.count(t[3 + i])) return err(PARTIR_E_SHAPE, "line %zu: unknown value '%s'", ln + 1, t[3 + i].c_str());
          op.in.push_back(by_name[t[3 + i]]);
        }
        const Value& a = values[op.in[0]];
        int64_t r = a.dim[0], c = a.dim[1];
        if (kind == "matmul") {
          const Value& b = values[op.in[1]];
          if (a.dim[1] != b.dim[0])
            return err(PARTIR_E_SHAPE, "line %zu: matmul %lldx%lld . %lldx%lld", ln + 1, (long long)a.dim[0],
                       (long long)a.dim[1], (long long)b.dim[0], (long long)b.dim[1]);
          c = b.dim[1];
        } else if (kind == "add") {
          const Value& b = values[op.in[1]];
          if (a.dim[0] != b.dim[0] || a.dim[1] != b.dim[1]) return err(PARTIR_E_SHAPE, "line %zu: add of different shapes", ln + 1);
        }
        op.out = (int)values.size();
        by_name[t[0]] = op.out;
        values.push_back(Value{t[0], {r, c}, (int)ops.size()});
        ops.push_back(op);
      } else {
        return err(PARTIR_E_SHAPE, "line %zu: cannot parse '%s'", ln + 1, ls[ln].c_str());
      }
    }
    const size_t na = axes.size();
    vtile.assign(values.size(), std::vector<int>(na, NONE));
    vslice.assign(values.size(), std::vector<int>(na, NONE));
    loop.assign(ops.size(), std::vector<int>(na, NONE));
    order.assign(ops.size(), {});
    slice.resize(ops.size());
    for (size_t o = 0; o < ops.size(); ++o) slice[o].assign(ops[o].in.size(), std::vector<int>(na, NONE));
    return Error{PARTIR_OK, ""};
  }

  // Product of the sizes of the axes that split dim d of operand `i` of op o,
  // counting axis `extra` too (TSlice: the dim must divide exactly).
  bool divisible_operand(int o, int i, int d, int extra) const {
    int64_t parts = axes[extra].size;
    for (size_t a = 0; a < axes.size(); ++a)
      if ((int)a != extra && slice[o][i][a] == d) parts *= axes[a].size;
    return values[ops[o].in[i]].dim[d] % parts == 0;
  }

  bool divisible_value(int v, int d, int extra) const {
    int64_t parts = axes[extra].size;
    for (size_t a = 0; a < axes.size(); ++a)
      if ((int)a != extra && vtile[v][a] == d) parts *= axes[a].size;
    return values[v].dim[d] % parts == 0;
  }

  bool applicable(int o, int a, const Entry& e) const {
    for (size_t i = 0; i < e.in.size(); ++i)
      if (e.in[i] != NONE && !divisible_operand(o, (int)i, e.in[i], a)) return false;
    if (e.out >= 0 && !divisible_value(ops[o].out, e.out, a)) return false;
    return true;
  }

  // dims along which the result of op o is used sliced on axis a
  std::set<int> sliced_uses(int o, int a) const {
    std::set<int> d;
    const int v = ops[o].out;
    if (vslice[v][a] != NONE) d.insert(vslice[v][a]);
    for (size_t c = 0; c < ops.size(); ++c) {
      if (loop[c][a] == NONE) continue;
      for (size_t i = 0; i < ops[c].in.size(); ++i)
        if (ops[c].in[i] == v && slice[c][i][a] != NONE) d.insert(slice[c][i][a]);
    }
    return d;
  }

  void apply(int o, int a, const Entry& e, const char* how) {
    loop[o][a] = e.out;
    order[o].push_back(a);
    for (size_t i = 0; i < e.in.size(); ++i) slice[o][i][a] = e.in[i];
    const int v = ops[o].out;
    if (e.out >= 0 && vtile[v][a] == NONE) vtile[v][a] = e.out;
    std::string act = e.out == SUM ? "#sum" : "#tile<" + std::to_string(e.out) + ">";
    actions.push_back(std::string("rewrite ") + values[v].name + " " + axes[a].name + " " + act + " " + how);
  }

  // One propagation step for op o on axis a; true if it introduced a loop.
  bool step(int o, int a) {
    if (loop[o][a] != NONE || conflicts.count({o, a})) return false;
    const auto& entries = tmr(ops[o].kind);
    const Op& op = ops[o];
    std::vector<int> full;
    for (size_t k = 0; k < entries.size(); ++k) {
      const Entry& e = entries[k];
      bool ok = true, any = false;
      for (size_t i = 0; i < e.in.size(); ++i) {
        if (e.in[i] == NONE) continue;
        any = true;
        if (vtile[op.in[i]][a] != e.in[i]) ok = false;
      }
      if (ok && any) full.push_back((int)k);
    }
    const std::set<int> uses = sliced_uses(o, a);
    std::vector<int> cand = full;
    for (size_t k = 0; k < entries.size(); ++k)
      if (entries[k].out >= 0 && uses.count(entries[k].out) &&
          std::find(cand.begin(), cand.end(), (int)k) == cand.end())
        cand.push_back((int)k);
    std::vector<int> fit;
    for (int k : cand)
      if (applicable(o, a, entries[k])) fit.push_back(k);
    if (fit.size() == 1) {
      const bool fwd = std::find(full.begin(), full.end(), fit[0]) != full.end();
      apply(o, a, entries[fit[0]], fwd ? "(forward)" : "(backward)");
      return true;
    }
    if (fit.size() > 1) {
      conflicts.insert({o, a});
      actions.push_back("conflict " + values[op.out].name + " " + axes[a].name + " " + std::to_string(fit.size()) +
                        " entries match");
      return false;
    }
    // inference from a partial match
    std::vector<int> part;
    for (size_t k = 0; k < entries.size(); ++k) {
      const Entry& e = entries[k];
      bool hit = false, clash = false;
      for (size_t i = 0; i < e.in.size(); ++i) {
        if (e.in[i] == NONE) continue;
        const int t = vtile[op.in[i]][a];
        if (t == e.in[i]) hit = true;
        else if (t != NONE) clash = true;
      }
      if (hit && !clash && applicable(o, a, e)) part.push_back((int)k);
    }
    if (part.size() == 1) {
      apply(o, a, entries[part[0]], "(inference)");
      return true;
    }
    if (part.size() > 1) {
      conflicts.insert({o, a});
      actions.push_back("conflict " + values[op.out].name + " " + axes[a].name + " " + std::to_string(part.size()) +
                        " partial matches");
    }
    return false;
  }

  void propagate() {
    actions.push_back("propagate");
    for (bool changed = true; changed;) {
      changed = false;
      for (size_t a = 0; a < axes.size(); ++a) {
        for (size_t o = 0; o < ops.size(); ++o) changed |= step((int)o, (int)a);
        for (size_t o = ops.size(); o-- > 0;) changed |= step((int)o, (int)a);
      }
    }
  }

  Error tile(const std::string& name, int d, const std::string& axis) {
    if (!by_name.count(name)) return err(PARTIR_E_SHAPE, "tile: unknown value '%s'", name.c_str());
    const int a = axis_index(axis);
    if (a < 0) return err(PARTIR_E_AXIS, "tile: unknown axis '%s'", axis.c_str());
    if (d < 0 || d > 1) return err(PARTIR_E_AXIS, "tile: dim %d of a 2-D value", d);
    const int v = by_name[name];
    actions.push_back("tile " + name + " " + std::to_string(d) + " " + axis);
    if (vtile[v][a] != NONE && vtile[v][a] != d)
      return err(PARTIR_E_AXIS, "tile: '%s' is already tiled along dim %d on axis '%s'", name.c_str(), vtile[v][a], axis.c_str());
    if (!divisible_value(v, d, a))
      return err(PARTIR_E_DIVISIBILITY, "tile: dim %d of '%s' (%lld) is not divisible by the axes that split it", d,
                 name.c_str(), (long long)values[v].dim[d]);
    vtile[v][a] = d;
    vslice[v][a] = d;
    return Error{PARTIR_OK, ""};
  }

  Error run_schedule(const char* text) {
    const auto ls = lines_of(text);
    for (size_t ln = 0; ln < ls.size(); ++ln) {
      const auto t = split_ws(ls[ln]);
      if (t.empty()) continue;
      if (t[0] == "partition" && t.size() >= 3) {       // ManualPartition({name: dim, ...}, axis)
        for (size_t i = 2; i < t.size(); ++i) {
          const size_t c = t[i].find(':');
          int64_t d;
          if (c == std::string::npos || !parse_int(t[i].substr(c + 1), d))
            return err(PARTIR_E_SHAPE, "schedule line %zu: expected name:dim, got '%s'", ln + 1, t[i].c_str());
          Error e = tile(t[i].substr(0, c), (int)d, t[1]);
          if (e.status) return e;
        }
        propagate();
      } else if (t[0] == "tile" && t.size() == 4) {     // a bare action
        int64_t d;
        if (!parse_int(t[2], d)) return err(PARTIR_E_SHAPE, "schedule line %zu: bad dim", ln + 1);
        Error e = tile(t[1], (int)d, t[3]);
        if (e.status) return e;
      } else if (t[0] == "propagate" && t.size() == 1) {
        propagate();
      } else {
        return err(PARTIR_E_SHAPE, "schedule line %zu: cannot parse '%s'", ln + 1, ls[ln].c_str());
      }
    }
    return Error{PARTIR_OK, ""};
  }

  static std::string act_name(int x) { return x == SUM ? "sum" : "tile" + std::to_string(x); }

  int axis_of(int o, int action) const {
    for (int a : order[o])
      if (loop[o][a] == action) return a;
    return -1;
  }

  // libpartir entry points for the nests the planner recognises
  std::vector<std::string> calls() const {
    std::vector<std::string> out;
    std::vector<bool> used(ops.size(), false);
    auto users = [&](int v) {
      std::vector<int> u;
      for (size_t c = 0; c < ops.size(); ++c)
        for (int x : ops[c].in)
          if (x == v) u.push_back((int)c);
      return u;
    };
    // Megatron MLP block: y = matmul(gelu(matmul(x, w1)), w2) with the batch
    // axis #tile<0> on all three ops and the model axis #tile<1>, #tile<1>, #sum
    for (size_t o = 0; o < ops.size(); ++o) {
      if (ops[o].kind != "matmul") continue;
      const auto u1 = users(ops[o].out);
      if (u1.size() != 1 || ops[u1[0]].kind != "gelu") continue;
      const int g = u1[0];
      const auto u2 = users(ops[g].out);
      if (u2.size() != 1 || ops[u2[0]].kind != "matmul" || ops[u2[0]].in[0] != ops[g].out) continue;
      const int o2 = u2[0];
      int rb = 1, rm = 1, ab = -1, am = -1;
      bool ok = true;
      for (size_t a = 0; a < axes.size() && ok; ++a) {
        const int l1 = loop[o][a], lg = loop[g][a], l2 = loop[o2][a];
        if (l1 == NONE && lg == NONE && l2 == NONE) continue;
        if (l1 == 0 && lg == 0 && l2 == 0 && rb == 1) rb = axes[a].size, ab = (int)a;
        else if (l1 == 1 && lg == 1 && l2 == SUM && rm == 1) rm = axes[a].size, am = (int)a;
        else ok = false;
      }
      if (!ok) continue;
      used[o] = used[g] = used[o2] = true;
      // BP + MP + Z3 with the activations sharded over the model axis: the
      // weights tiled over the batch axis (w1 dim 0, w2 dim 1) and x tiled
      // over the model axis on dim 0 are all used whole (all_gathers) -> the
      // entry point on device-local arrays
      const int x = ops[o].in[0], w1 = ops[o].in[1], w2 = ops[o2].in[1];
      const bool z3 = ab >= 0 && am >= 0 && vtile[w1][ab] == 0 && vtile[w2][ab] == 1;
      const bool sp = am >= 0 && vtile[x][am] == 0;
      out.push_back(std::string(z3 && sp ? "call partir_mlp_block_sharded " : "call partir_mlp_block ") +
                    values[ops[o2].out].name + " R_batch=" + std::to_string(rb) + " R_model=" + std::to_string(rm) +
                    " ops=" + values[ops[o].out].name + "," + values[ops[g].out].name + "," +
                    values[ops[o2].out].name);
    }
    // a single partitioned matmul: at most one #tile and one #sum loop of one size
    for (size_t o = 0; o < ops.size(); ++o) {
      if (used[o] || ops[o].kind != "matmul") continue;
      std::string tile = "none", sum = "none";
      int R = 1, ntile = 0, nsum = 0;
      bool same = true;
      for (int a : order[o]) {
        const int l = loop[o][a];
        if (l == SUM) ++nsum, sum = "K";
        else ++ntile, tile = l == 0 ? "M" : "N";
        if (R != 1 && R != axes[a].size) same = false;
        R = axes[a].size;
      }
      if (ntile <= 1 && nsum <= 1 && same)
        out.push_back("call partir_loop_matmul " + values[ops[o].out].name + " tile=" + tile + " sum=" + sum +
                      " R=" + std::to_string(R));
      else
        out.push_back("nest " + values[ops[o].out].name + " (no single entry point: a host loop over the outer axes)");
    }
    return out;
  }

  std::string report() const {
    std::string s;
    for (const auto& a : actions) s += "action " + a + "\n";
    for (size_t o = 0; o < ops.size(); ++o) {
      s += "loop " + values[ops[o].out].name + " " + ops[o].kind;
      if (order[o].empty()) s += " none";
      for (int a : order[o]) s += " " + axes[a].name + ":" + act_name(loop[o][a]);
      s += "\n";
      for (size_t i = 0; i < ops[o].in.size(); ++i) {
        std::string sl;
        for (int a : order[o])
          if (slice[o][i][a] != NONE) sl += " " + axes[a].name + ":" + std::to_string(slice[o][i][a]);
        if (!sl.empty()) s += "operand " + values[ops[o].out].name + " " + std::to_string(i) + " " + values[ops[o].in[i]].name + sl + "\n";
        // an operand tiled on an axis but not sliced along that dim by this op
        // is used whole (an all_gather in the SPMD lowering) or resliced
        for (size_t a = 0; a < axes.size(); ++a) {
          const int t = vtile[ops[o].in[i]][a];
          if (t == NONE || slice[o][i][a] == t) continue;
          s += std::string(slice[o][i][a] == NONE ? "gather " : "reshard ") + values[ops[o].out].name + " " +
               values[ops[o].in[i]].name + " " + axes[a].name + "\n";
        }
      }
    }
    for (size_t v = 0; v < values.size(); ++v) {
      std::string t;
      for (size_t a = 0; a < axes.size(); ++a)
        if (vtile[v][a] != NONE) t += " " + axes[a].name + ":" + std::to_string(vtile[v][a]);
      s += "value " + values[v].name + (t.empty() ? " replicated" : t) + "\n";
    }
    for (const auto& c : calls()) s += c + "\n";
    return s;
  }
};

}  // namespace planner
}  // namespace partir

namespace partir {
void set_last_error(const std::string& msg);   // the C ABI's thread-local message
}

extern "C" int partir_propagate(const char* program, const char* schedule, char* out, size_t out_len,
                                size_t* needed) {
  using namespace partir::planner;
  if (!program || !schedule) {
    partir::set_last_error("PARTIR_E_NULL: program and schedule must be non-NULL");
    return PARTIR_E_NULL;
  }
  Planner p;
  Error e = p.parse_program(program);
  if (e.status == PARTIR_OK) e = p.run_schedule(schedule);
  if (e.status != PARTIR_OK) {
    partir::set_last_error(std::string(partir_status_string(e.status)) + ": " + e.msg);
    return e.status;
  }
  const std::string r = p.report();
  if (needed) *needed = r.size() + 1;
  if (!out || out_len < r.size() + 1) {
    partir::set_last_error("PARTIR_E_WORKSPACE: output buffer of " + std::to_string(out_len) + " bytes, need " +
                           std::to_string(r.size() + 1));
    return PARTIR_E_WORKSPACE;
  }
  memcpy(out, r.c_str(), r.size() + 1);
  return PARTIR_OK;
}
