// ea_exprog.cpp -- exchange programs (Section 5.2): the ExProg text format,
// the closure and validity of Definition "Closure; validity", memberships of
// partitions declared by size, the naive valid program that gathers the
// atoms of every required aggregate at its targets (Section 5.4), and a
// simulator of a full point-to-point mesh (every GPU pair linked, as xGMI
// connects an 8-GPU MI355X node) that gives a valid program its completion
// time.
#include <algorithm>
#include <cctype>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "ea_internal.h"

namespace ea {
namespace {

using Agg = std::vector<int>;  // sorted atom ids

struct Target {
  bool part = false;
  int id = 0;  // site, or partition index
};

struct Action {
  Agg agg;
  std::vector<Target> src;
  std::vector<std::vector<Target>> hops;  // destination lists, in order
  std::string text;
};

struct Part {
  std::string name;
  int size = 0;
  bool by_size = false;
  std::vector<int> members;
};

struct Prog {
  std::vector<int> gpus;
  bool implicit_gpus = false;  // no GPUS declaration: every site named is a GPU
  std::vector<std::string> atom_name;
  std::vector<double> atom_bytes;
  std::map<std::string, int> atom_id;
  std::vector<Part> parts;
  std::vector<std::pair<int, int>> ins;  // (atom, site)
  std::vector<std::pair<Agg, std::vector<Target>>> outs;
  std::vector<Action> acts;
  std::string decl_text;  // the declarations, as written
};

std::string trim(const std::string& s) {
  size_t a = 0, b = s.size();
  while (a < b && isspace((unsigned char)s[a])) ++a;
  while (b > a && isspace((unsigned char)s[b - 1])) --b;
  return s.substr(a, b - a);
}

std::vector<std::string> split(const std::string& s, char sep) {
  std::vector<std::string> out;
  std::string cur;
  for (char c : s) {
    if (c == sep) {
      out.push_back(cur);
      cur.clear();
    } else {
      cur += c;
    }
  }
  out.push_back(cur);
  return out;
}

bool parse_int(const std::string& t, int* v) {
  const std::string s = trim(t);
  if (s.empty()) return false;
  for (char c : s)
    if (!isdigit((unsigned char)c)) return false;
  *v = atoi(s.c_str());
  return true;
}

int site_of(Prog& p, const std::string& tok, Target* t) {
  int v;
  const std::string s = trim(tok);
  if (parse_int(s, &v)) {
    if (std::find(p.gpus.begin(), p.gpus.end(), v) == p.gpus.end()) {
      if (!p.implicit_gpus) return fail(EA_ERR_SPEC, "ExProg: site %d is not among the GPUS", v);
      p.gpus.push_back(v);
    }
    *t = Target{false, v};
    return EA_OK;
  }
  for (size_t i = 0; i < p.parts.size(); ++i)
    if (p.parts[i].name == s) {
      *t = Target{true, (int)i};
      return EA_OK;
    }
  return fail(EA_ERR_SPEC, "ExProg: unknown site or partition '%s'", s.c_str());
}

int targets_of(Prog& p, const std::string& list, std::vector<Target>* out) {
  out->clear();
  for (const std::string& tok : split(list, ',')) {
    Target t;
    const int e = site_of(p, tok, &t);
    if (e) return e;
    out->push_back(t);
  }
  return EA_OK;
}

int agg_of(Prog& p, const std::string& text, Agg* out) {
  out->clear();
  for (const std::string& tok : split(text, '+')) {
    const std::string a = trim(tok);
    auto it = p.atom_id.find(a);
    if (it == p.atom_id.end()) return fail(EA_ERR_SPEC, "ExProg: unknown atom '%s'", a.c_str());
    out->push_back(it->second);
  }
  std::sort(out->begin(), out->end());
  if (std::adjacent_find(out->begin(), out->end()) != out->end())
    return fail(EA_ERR_SPEC, "ExProg: atom repeated in '%s'", trim(text).c_str());
  return EA_OK;
}

double parse_size(const std::string& s) {  // "(size: 1.5 GB)"
  const size_t c = s.find(':');
  const std::string body = trim(s.substr(c == std::string::npos ? 0 : c + 1));
  char* end = nullptr;
  const double v = strtod(body.c_str(), &end);
  std::string unit = trim(std::string(end));
  if (!unit.empty() && unit.back() == ')') unit.pop_back();
  unit = trim(unit);
  const double scale = unit == "KB" ? 1e3 : unit == "MB" ? 1e6 : unit == "B" ? 1.0 : 1e9;
  return v * scale;
}

const char* kKeys[] = {"GPUS:", "PARTITIONS:", "IN:", "OUT:"};

int key_of(const std::string& line) {
  const std::string s = trim(line);
  for (int k = 0; k < 4; ++k)
    if (s.compare(0, strlen(kKeys[k]), kKeys[k]) == 0) return k;
  return -1;
}

int parse(const char* text, Prog* p) {
  std::string sect[4];
  std::string body;
  int cur = -1;
  bool in_body = false, any_decl = false;
  std::string decl;
  for (const std::string& raw : split(text, '\n')) {
    const std::string line = trim(raw);
    const int k = key_of(line);
    if (k >= 0) {
      cur = k;
      in_body = false;
      any_decl = true;
      sect[k] += " " + line.substr(strlen(kKeys[k])) + ";";
      decl += raw + "\n";
      continue;
    }
    if (line.empty()) {
      if (any_decl) in_body = true;
      cur = -1;
      continue;
    }
    if (cur >= 0 && !in_body) {
      sect[cur] += " " + line + ";";
      decl += raw + "\n";
    } else {
      body += line + ";";
    }
  }
  p->decl_text = decl;
  // GPUS (default: every site named anywhere is an error without it)
  for (const std::string& tok : split(sect[0], ',')) {
    for (const std::string& t2 : split(tok, ';')) {
      int v;
      if (trim(t2).empty()) continue;
      if (!parse_int(t2, &v)) return fail(EA_ERR_SPEC, "ExProg: bad GPU '%s'", trim(t2).c_str());
      p->gpus.push_back(v);
    }
  }
  p->implicit_gpus = p->gpus.empty();
  // PARTITIONS: name {size n} | name {a, b, ...}
  {
    std::string s = sect[1];
    size_t i = 0;
    while (true) {
      const size_t lb = s.find('{', i);
      if (lb == std::string::npos) break;
      const size_t rb = s.find('}', lb);
      if (rb == std::string::npos) return fail(EA_ERR_SPEC, "ExProg: unclosed partition");
      std::string name = trim(s.substr(i, lb - i));
      while (!name.empty() && name.front() == ';') name = trim(name.substr(1));
      const std::string inner = trim(s.substr(lb + 1, rb - lb - 1));
      Part pt;
      pt.name = name;
      if (name.empty()) return fail(EA_ERR_SPEC, "ExProg: unnamed partition");
      if (inner.compare(0, 4, "size") == 0) {
        pt.by_size = true;
        if (!parse_int(inner.substr(4), &pt.size) || pt.size < 1)
          return fail(EA_ERR_SPEC, "ExProg: partition %s: bad size", name.c_str());
      } else {
        for (const std::string& tok : split(inner, ',')) {
          int v;
          if (!parse_int(tok, &v)) return fail(EA_ERR_SPEC, "ExProg: partition %s: bad member", name.c_str());
          pt.members.push_back(v);
        }
        pt.size = (int)pt.members.size();
      }
      p->parts.push_back(pt);
      i = rb + 1;
    }
    for (const Part& pt : p->parts)
      for (int m : pt.members) {
        Target t;
        const int e = site_of(*p, std::to_string(m), &t);
        if (e) return e;
      }
  }
  // IN: atom @ site (size: ...)
  for (const std::string& st : split(sect[2], ';')) {
    std::string s = trim(st);
    if (s.empty()) continue;
    double bytes = 1e9;
    const size_t lp = s.find('(');
    if (lp != std::string::npos) {
      bytes = parse_size(s.substr(lp + 1));
      s = trim(s.substr(0, lp));
    }
    const size_t at = s.find('@');
    if (at == std::string::npos) return fail(EA_ERR_SPEC, "ExProg: IN '%s' has no '@'", s.c_str());
    const std::string name = trim(s.substr(0, at));
    if (name.empty() || name.find('+') != std::string::npos)
      return fail(EA_ERR_SPEC, "ExProg: IN '%s' must place one atom", s.c_str());
    Target t;
    int e = site_of(*p, s.substr(at + 1), &t);
    if (e) return e;
    if (t.part) return fail(EA_ERR_SPEC, "ExProg: IN places atoms at GPUs");
    if (p->atom_id.count(name)) return fail(EA_ERR_SPEC, "ExProg: atom %s placed twice", name.c_str());
    p->atom_id[name] = (int)p->atom_name.size();
    p->atom_name.push_back(name);
    p->atom_bytes.push_back(bytes);
    p->ins.push_back({p->atom_id[name], t.id});
  }
  // OUT: aggregate @ targets
  for (const std::string& st : split(sect[3], ';')) {
    const std::string s = trim(st);
    if (s.empty()) continue;
    const size_t at = s.find('@');
    if (at == std::string::npos) return fail(EA_ERR_SPEC, "ExProg: OUT '%s' has no '@'", s.c_str());
    Agg a;
    std::vector<Target> ts;
    int e = agg_of(*p, s.substr(0, at), &a);
    if (!e) e = targets_of(*p, s.substr(at + 1), &ts);
    if (e) return e;
    p->outs.push_back({a, ts});
  }
  // body: X @ sources [-> destinations ...]
  for (const std::string& st : split(body, ';')) {
    const std::string s = trim(st);
    if (s.empty()) continue;
    Action act;
    act.text = s;
    std::vector<std::string> parts;
    size_t i = 0;
    while (true) {
      const size_t ar = s.find("->", i);
      parts.push_back(s.substr(i, ar == std::string::npos ? std::string::npos : ar - i));
      if (ar == std::string::npos) break;
      i = ar + 2;
    }
    const size_t at = parts[0].find('@');
    if (at == std::string::npos) return fail(EA_ERR_SPEC, "ExProg: action '%s' has no '@'", s.c_str());
    int e = agg_of(*p, parts[0].substr(0, at), &act.agg);
    if (!e) e = targets_of(*p, parts[0].substr(at + 1), &act.src);
    for (size_t h = 1; !e && h < parts.size(); ++h) {
      std::vector<Target> d;
      e = targets_of(*p, parts[h], &d);
      act.hops.push_back(d);
    }
    if (e) return e;
    p->acts.push_back(act);
  }
  // partitions: disjoint, together covering the GPUs
  int total = 0;
  std::set<int> seen;
  for (const Part& pt : p->parts) {
    total += pt.size;
    for (int m : pt.members)
      if (!seen.insert(m).second) return fail(EA_ERR_SPEC, "ExProg: site %d in two partitions", m);
  }
  if (!p->parts.empty() && total != (int)p->gpus.size())
    return fail(EA_ERR_SPEC, "ExProg: partitions hold %d sites, not the %d GPUS", total, (int)p->gpus.size());
  std::sort(p->gpus.begin(), p->gpus.end());
  return EA_OK;
}

std::vector<int> sites(const Prog& p, const std::vector<Target>& ts, const std::vector<std::vector<int>>& mem) {
  std::vector<int> out;
  for (const Target& t : ts) {
    if (!t.part) out.push_back(t.id);
    else out.insert(out.end(), mem[(size_t)t.id].begin(), mem[(size_t)t.id].end());
  }
  return out;
}

// do aggregates present at a site partition X (an exact cover by subsets)?
// Larger parts are tried first; the cover found goes to *cover if given.
bool covers(const std::set<Agg>& here, const Agg& x, std::vector<const Agg*>* cover = nullptr) {
  if (here.count(x)) {
    if (cover) cover->assign(1, &*here.find(x));
    return true;
  }
  std::vector<const Agg*> cand;
  for (const Agg& a : here)
    if (std::includes(x.begin(), x.end(), a.begin(), a.end())) cand.push_back(&a);
  std::stable_sort(cand.begin(), cand.end(), [](const Agg* a, const Agg* b) { return a->size() > b->size(); });
  std::vector<const Agg*> chosen;
  std::vector<char> used(x.size(), 0);
  auto pos = [&](int atom) { return (size_t)(std::lower_bound(x.begin(), x.end(), atom) - x.begin()); };
  auto rec = [&](auto&& self) -> bool {
    size_t first = 0;
    while (first < x.size() && used[first]) ++first;
    if (first == x.size()) return true;
    for (const Agg* a : cand) {
      if (!std::binary_search(a->begin(), a->end(), x[first])) continue;
      bool free_all = true;
      for (int at : *a) free_all &= !used[pos(at)];
      if (!free_all) continue;
      for (int at : *a) used[pos(at)] = 1;
      chosen.push_back(a);
      if (self(self)) return true;
      chosen.pop_back();
      for (int at : *a) used[pos(at)] = 0;
    }
    return false;
  };
  const bool ok_cover = rec(rec);
  if (ok_cover && cover) *cover = chosen;
  return ok_cover;
}

// closure and validity for one membership of the partitions; the closure
// goes to *closure if given
bool check(const Prog& p, const std::vector<std::vector<int>>& mem, std::string* why,
           std::map<int, std::set<Agg>>* closure = nullptr) {
  std::map<int, std::set<Agg>> state;
  for (const auto& in : p.ins) state[in.second].insert(Agg{in.first});
  // (action, source site) pairs; fired when enabled, to a fixed point
  std::vector<std::pair<int, int>> todo;
  for (size_t a = 0; a < p.acts.size(); ++a)
    for (int s : sites(p, p.acts[a].src, mem)) todo.push_back({(int)a, s});
  std::vector<char> fired(todo.size(), 0);
  for (bool changed = true; changed;) {
    changed = false;
    for (size_t i = 0; i < todo.size(); ++i) {
      if (fired[i]) continue;
      const Action& act = p.acts[(size_t)todo[i].first];
      if (!covers(state[todo[i].second], act.agg)) continue;
      fired[i] = 1;
      changed = true;
      state[todo[i].second].insert(act.agg);
      for (const auto& hop : act.hops)
        for (int d : sites(p, hop, mem)) state[d].insert(act.agg);
    }
  }
  if (closure) *closure = state;
  for (size_t i = 0; i < todo.size(); ++i)
    if (!fired[i]) {
      *why = "action '" + p.acts[(size_t)todo[i].first].text + "' is never enabled at site " +
             std::to_string(todo[i].second);
      return false;
    }
  for (const auto& req : p.outs)
    for (int s : sites(p, req.second, mem))
      if (!state[s].count(req.first)) {
        std::string name;
        for (int a : req.first) name += (name.empty() ? "" : "+") + p.atom_name[(size_t)a];
        *why = "OUT " + name + " is not materialised at site " + std::to_string(s);
        return false;
      }
  return true;
}

// memberships of the partitions declared by size, lexicographic order; fn
// returns true to stop
template <class F>
void memberships(const Prog& p, F&& fn) {
  std::vector<std::vector<int>> mem(p.parts.size());
  std::vector<int> free;
  std::set<int> taken;
  for (size_t i = 0; i < p.parts.size(); ++i)
    if (!p.parts[i].by_size) {
      mem[i] = p.parts[i].members;
      taken.insert(p.parts[i].members.begin(), p.parts[i].members.end());
    }
  for (int g : p.gpus)
    if (!taken.count(g)) free.push_back(g);
  std::vector<char> used(free.size(), 0);
  bool stop = false;
  auto rec = [&](auto&& self, size_t part) -> void {
    if (stop) return;
    while (part < p.parts.size() && !p.parts[part].by_size) ++part;
    if (part == p.parts.size()) {
      stop = fn(mem);
      return;
    }
    // choose size-many unused free sites in increasing order
    std::vector<int>& m = mem[part];
    auto pick = [&](auto&& pk, size_t from) -> void {
      if (stop) return;
      if ((int)m.size() == p.parts[part].size) {
        self(self, part + 1);
        return;
      }
      for (size_t j = from; j < free.size(); ++j) {
        if (used[j]) continue;
        used[j] = 1;
        m.push_back(free[j]);
        pk(pk, j + 1);
        m.pop_back();
        used[j] = 0;
        if (stop) return;
      }
    };
    pick(pick, 0);
  };
  rec(rec, 0);
}

// Completion time of a valid program on a full mesh: dataflow semantics
// (an action starts once its aggregate's parts are present at its source;
// every eligible action proceeds concurrently).  An action is a pipeline of
// stages: the local aggregation of its parts (reading them and writing the
// aggregate at the GPU's memory bandwidth; none when the aggregate is
// present as one piece), then each hop's transfers, one per destination,
// each on the directed link between the two GPUs.  Stages that share a
// resource (a GPU's memory, a directed link) share its bandwidth equally.
// An aggregate's size is its largest atom's.
double simulate(const Prog& p, const std::vector<std::vector<int>>& mem, double link_bps, double hbm_bps) {
  struct Task {
    int act, site;              // action and source site
    int stage = 0;              // 0 aggregation, 1.. hop transfers
    std::vector<int> from, to;  // current hop: transfers (from[i] -> to[i])
    std::vector<double> left;   // bytes left per transfer (stage >= 1), or [0]: the aggregation
    bool started = false, done = false;
  };
  std::map<int, std::set<Agg>> state;
  for (const auto& in : p.ins) state[in.second].insert(Agg{in.first});
  auto size_of = [&](const Agg& a) {
    double m = 0;
    for (int x : a) m = std::max(m, p.atom_bytes[(size_t)x]);
    return m;
  };
  std::vector<Task> tasks;
  for (size_t a = 0; a < p.acts.size(); ++a)
    for (int s : sites(p, p.acts[a].src, mem)) {
      Task t;
      t.act = (int)a;
      t.site = s;
      tasks.push_back(t);
    }
  // the aggregation reads the parts of one cover (larger parts first) and
  // writes the aggregate; nothing when it is present as one piece
  auto parts_bytes = [&](const Agg& x, int s) {
    if (state[s].count(x)) return 0.0;
    std::vector<const Agg*> cover;
    covers(state[s], x, &cover);
    double bytes = size_of(x);
    for (const Agg* a : cover) bytes += size_of(*a);
    return bytes;
  };
  auto start_hop = [&](Task& t, int hop) {
    const Action& act = p.acts[(size_t)t.act];
    t.stage = hop + 1;
    t.from.clear();
    t.to.clear();
    t.left.clear();
    const std::vector<int> srcs = hop == 0 ? std::vector<int>{t.site} : sites(p, act.hops[(size_t)hop - 1], mem);
    for (int f : srcs)
      for (int d : sites(p, act.hops[(size_t)hop], mem))
        if (d != f) {
          t.from.push_back(f);
          t.to.push_back(d);
          t.left.push_back(size_of(act.agg));
        }
  };
  double now = 0;
  for (int guard = 0; guard < 1 << 22; ++guard) {
    // start every eligible action
    for (Task& t : tasks) {
      if (t.started) continue;
      const Action& act = p.acts[(size_t)t.act];
      if (!covers(state[t.site], act.agg)) continue;
      t.started = true;
      t.stage = 0;
      t.left = {parts_bytes(act.agg, t.site)};
    }
    // advance stages that have nothing left
    bool moved = true;
    while (moved) {
      moved = false;
      for (Task& t : tasks) {
        if (!t.started || t.done) continue;
        bool empty = true;
        for (double b : t.left) empty &= b <= 0;
        if (!empty) continue;
        const Action& act = p.acts[(size_t)t.act];
        if (t.stage == 0) state[t.site].insert(act.agg);
        else
          for (int d : t.to) state[d].insert(act.agg);
        if (t.stage < (int)act.hops.size()) {
          start_hop(t, t.stage);
        } else {
          t.done = true;
        }
        moved = true;
      }
    }
    // active resource users: GPU memory (stage 0) and directed links
    std::map<std::pair<int, int>, int> users;  // (from, to) link; (-1 - gpu, 0) memory
    for (const Task& t : tasks) {
      if (!t.started || t.done) continue;
      if (t.stage == 0) {
        if (t.left[0] > 0) ++users[{-1 - t.site, 0}];
      } else {
        for (size_t i = 0; i < t.to.size(); ++i)
          if (t.left[i] > 0) ++users[{t.from[i], t.to[i]}];
      }
    }
    if (users.empty()) {
      bool all_done = true;
      for (const Task& t : tasks) all_done &= t.done;
      if (all_done) return now;
      bool any_new = false;  // something may have become eligible
      for (const Task& t : tasks)
        if (!t.started && covers(state[t.site], p.acts[(size_t)t.act].agg)) any_new = true;
      if (!any_new) return -1;  // stuck: not a valid program
      continue;
    }
    auto rate = [&](const std::pair<int, int>& r) {
      return (r.first < 0 ? hbm_bps : link_bps) / users[r];
    };
    double dt = 1e300;
    for (const Task& t : tasks) {
      if (!t.started || t.done) continue;
      if (t.stage == 0) {
        if (t.left[0] > 0) dt = std::min(dt, t.left[0] / rate({-1 - t.site, 0}));
      } else {
        for (size_t i = 0; i < t.to.size(); ++i)
          if (t.left[i] > 0) dt = std::min(dt, t.left[i] / rate({t.from[i], t.to[i]}));
      }
    }
    for (Task& t : tasks) {
      if (!t.started || t.done) continue;
      if (t.stage == 0) {
        if (t.left[0] > 0) t.left[0] = std::max(0.0, t.left[0] - dt * rate({-1 - t.site, 0}));
      } else {
        for (size_t i = 0; i < t.to.size(); ++i)
          if (t.left[i] > 0) t.left[i] = std::max(0.0, t.left[i] - dt * rate({t.from[i], t.to[i]}));
      }
    }
    // finish the stage whose remainder is within rounding of zero
    for (Task& t : tasks)
      for (double& b : t.left)
        if (b > 0 && b < 1e-6) b = 0;
    now += dt;
  }
  return -1;
}

// ---- body synthesis (Section 5.4) ----------------------------------------
// Bodies are searched with concrete sites: an action is an aggregate, one
// source GPU and its hops' destination GPUs.
struct FAct {
  Agg agg;
  int src = 0;
  std::vector<std::vector<int>> hops;
  bool operator==(const FAct& o) const { return agg == o.agg && src == o.src && hops == o.hops; }
};

std::string agg_name(const Prog& p, const Agg& a) {
  std::string n;
  for (int x : a) n += (n.empty() ? "" : "+") + p.atom_name[(size_t)x];
  return n;
}

std::string render_act(const Prog& p, const FAct& f) {
  std::string t = agg_name(p, f.agg) + " @ " + std::to_string(f.src);
  for (const auto& h : f.hops) {
    t += " ->";
    for (size_t i = 0; i < h.size(); ++i) t += (i ? ", " : " ") + std::to_string(h[i]);
  }
  return t;
}

Prog with_body(const Prog& base, const std::vector<FAct>& body) {
  Prog q = base;
  q.acts.clear();
  for (const FAct& f : body) {
    Action a;
    a.agg = f.agg;
    a.src = {Target{false, f.src}};
    for (const auto& h : f.hops) {
      std::vector<Target> ts;
      for (int d : h) ts.push_back(Target{false, d});
      a.hops.push_back(ts);
    }
    a.text = render_act(base, f);
    q.acts.push_back(a);
  }
  return q;
}

// the naive valid program (Section 5.4): the atoms of every required
// aggregate go from their IN site to each target, which aggregates locally
std::vector<FAct> naive_body(const Prog& p, const std::vector<std::vector<int>>& mem) {
  std::vector<FAct> body;
  auto add = [&](const FAct& f) {
    if (std::find(body.begin(), body.end(), f) == body.end()) body.push_back(f);
  };
  std::vector<int> home(p.atom_name.size(), -1);
  for (const auto& in : p.ins) home[(size_t)in.first] = in.second;
  for (const auto& req : p.outs)
    for (int t : sites(p, req.second, mem)) {
      for (int a : req.first)
        if (home[(size_t)a] != t) add(FAct{Agg{a}, home[(size_t)a], {{t}}});
      if (req.first.size() > 1) add(FAct{req.first, t, {}});
    }
  return body;
}

// declarations with the memberships fixed and sizes kept exactly
std::string render_decls(const Prog& p, const std::vector<std::vector<int>>& mem) {
  std::string t = "GPUS: ";
  for (size_t i = 0; i < p.gpus.size(); ++i) t += (i ? ", " : "") + std::to_string(p.gpus[i]);
  t += "\n";
  if (!p.parts.empty()) {
    t += "PARTITIONS:";
    for (size_t i = 0; i < p.parts.size(); ++i) {
      t += " " + p.parts[i].name + " {";
      for (size_t j = 0; j < mem[i].size(); ++j) t += (j ? ", " : "") + std::to_string(mem[i][j]);
      t += "}";
    }
    t += "\n";
  }
  t += "IN: ";
  for (size_t i = 0; i < p.ins.size(); ++i) {
    char buf[64];
    snprintf(buf, sizeof(buf), " (size: %.17g B)", p.atom_bytes[(size_t)p.ins[i].first]);
    t += (i ? "; " : "") + p.atom_name[(size_t)p.ins[i].first] + " @ " + std::to_string(p.ins[i].second) + buf;
  }
  t += "\nOUT: ";
  for (size_t i = 0; i < p.outs.size(); ++i) {
    t += (i ? "; " : "") + agg_name(p, p.outs[i].first) + " @ ";
    for (size_t j = 0; j < p.outs[i].second.size(); ++j) {
      const Target& g = p.outs[i].second[j];
      t += (j ? ", " : "") + (g.part ? p.parts[(size_t)g.id].name : std::to_string(g.id));
    }
  }
  return t + "\n";
}

struct Rng {  // splitmix64
  uint64_t s;
  uint64_t next() {
    uint64_t z = (s += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  int below(int n) { return n <= 1 ? 0 : (int)(next() % (uint64_t)n); }
  double unit() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
};

// One random transformation of Section 5.4 applied to body; false when the
// drawn move does not apply.  Validity is checked by the caller.
bool transform(const Prog& p, const std::map<int, std::set<Agg>>& closure, std::vector<FAct>& b, Rng& rng) {
  if (b.empty()) return false;
  const int kind = rng.below(8);
  const int i = rng.below((int)b.size());
  FAct& a = b[(size_t)i];
  const int ng = (int)p.gpus.size();
  auto single_hop = [](const FAct& f) { return f.hops.size() == 1; };
  switch (kind) {
    case 0: {  // multicast fission: X @ s -> D1 u D2  =>  X @ s -> D1; X @ s -> D2
      if (!single_hop(a) || a.hops[0].size() < 2) return false;
      std::vector<int> d1, d2;
      for (int d : a.hops[0]) (rng.below(2) ? d1 : d2).push_back(d);
      if (d1.empty() || d2.empty()) return false;
      FAct other{a.agg, a.src, {d2}};
      a.hops[0] = d1;
      b.push_back(other);
      return true;
    }
    case 1: {  // multicast fusion (the reverse)
      if (!single_hop(a)) return false;
      for (size_t j = 0; j < b.size(); ++j)
        if ((int)j != i && single_hop(b[j]) && b[j].agg == a.agg && b[j].src == a.src) {
          for (int d : b[j].hops[0])
            if (std::find(a.hops[0].begin(), a.hops[0].end(), d) == a.hops[0].end()) a.hops[0].push_back(d);
          std::sort(a.hops[0].begin(), a.hops[0].end());
          b.erase(b.begin() + (long)j);
          return true;
        }
      return false;
    }
    case 2: {  // relay introduction: X @ s -> d  =>  X @ s -> r -> d
      if (!single_hop(a) || ng < 3) return false;
      const int d = a.hops[0][(size_t)rng.below((int)a.hops[0].size())];
      const int r = p.gpus[(size_t)rng.below(ng)];
      if (r == a.src || r == d) return false;
      FAct relay{a.agg, a.src, {{r}, {d}}};
      if (a.hops[0].size() == 1) {
        a = relay;
      } else {
        a.hops[0].erase(std::find(a.hops[0].begin(), a.hops[0].end(), d));
        b.push_back(relay);
      }
      return true;
    }
    case 3: {  // relay elimination: X @ s -> r -> d  =>  X @ s -> d
      if (a.hops.size() != 2 || a.hops[0].size() != 1) return false;
      a.hops = {a.hops[1]};
      return true;
    }
    case 4: {  // aggregation pushdown: X @ r -> s; Y @ r -> s  =>  X+Y @ r -> s
      if (!single_hop(a) || a.hops[0].size() != 1) return false;
      for (size_t j = 0; j < b.size(); ++j) {
        const FAct& o = b[j];
        if ((int)j == i || !single_hop(o) || o.hops[0] != a.hops[0] || o.src != a.src) continue;
        Agg u;
        std::set_union(a.agg.begin(), a.agg.end(), o.agg.begin(), o.agg.end(), std::back_inserter(u));
        if (u.size() != a.agg.size() + o.agg.size()) continue;  // not disjoint
        a.agg = u;
        b.erase(b.begin() + (long)j);
        return true;
      }
      return false;
    }
    case 5: {  // aggregation pullup: X+Y @ r -> s  =>  X @ r -> s; Y @ r -> s; X+Y @ s
      if (!single_hop(a) || a.hops[0].size() != 1 || a.agg.size() < 2) return false;
      Agg x, y;
      for (int at : a.agg) (rng.below(2) ? x : y).push_back(at);
      if (x.empty() || y.empty()) return false;
      const FAct local{a.agg, a.hops[0][0], {}};
      const FAct fy{y, a.src, a.hops};
      a.agg = x;
      b.push_back(fy);
      if (std::find(b.begin(), b.end(), local) == b.end()) b.push_back(local);
      return true;
    }
    case 6: {  // source substitution: draw X from another site holding it
      if (a.hops.empty()) return false;
      std::vector<int> holders;
      for (const auto& kv : closure)
        if (kv.first != a.src && kv.second.count(a.agg)) holders.push_back(kv.first);
      if (holders.empty()) return false;
      const int s2 = holders[(size_t)rng.below((int)holders.size())];
      a.src = s2;
      for (auto& h : a.hops) h.erase(std::remove(h.begin(), h.end(), s2), h.end());
      a.hops.erase(std::remove_if(a.hops.begin(), a.hops.end(), [](const std::vector<int>& h) { return h.empty(); }),
                   a.hops.end());
      return true;
    }
    default:  // deletion of an action (guarded by validity)
      b.erase(b.begin() + i);
      return true;
  }
}

// Search from the naive program of the best membership: seeded simulated
// annealing over the transformations, every candidate checked for validity
// and costed by the simulator.  Returns the best cost, or -1.
double synthesize(const Prog& p, double link_bps, double hbm_bps, int iters, uint64_t seed,
                  std::vector<std::vector<int>>* mem_out, std::vector<FAct>* body_out) {
  const int kMaxMemberships = 5040;
  double best = -1;
  int tried = 0;
  memberships(p, [&](const std::vector<std::vector<int>>& mem) {
    const std::vector<FAct> nb = naive_body(p, mem);
    const Prog q = with_body(p, nb);
    std::string why;
    if (check(q, mem, &why)) {
      const double c = simulate(q, mem, link_bps, hbm_bps);
      if (c >= 0 && (best < 0 || c < best)) {
        best = c;
        *mem_out = mem;
        *body_out = nb;
      }
    }
    return ++tried >= kMaxMemberships;
  });
  if (best < 0) return -1;
  const std::vector<std::vector<int>> mem = *mem_out;
  Rng rng{seed};
  std::vector<FAct> cur = *body_out;
  double cur_cost = best;
  std::map<int, std::set<Agg>> closure;
  std::string why;
  check(with_body(p, cur), mem, &why, &closure);
  for (int it = 0; it < iters; ++it) {
    const double temp = 0.02 * best * (1.0 - (double)it / iters);
    std::vector<FAct> cand = cur;
    if (!transform(p, closure, cand, rng)) continue;
    const Prog q = with_body(p, cand);
    std::map<int, std::set<Agg>> cl;
    if (!check(q, mem, &why, &cl)) continue;
    const double c = simulate(q, mem, link_bps, hbm_bps);
    if (c < 0) continue;
    if (c <= cur_cost || (temp > 0 && rng.unit() < std::exp((cur_cost - c) / temp))) {
      cur = cand;
      cur_cost = c;
      closure = cl;
      if (c < best - 1e-15 || (c <= best && cand.size() < body_out->size())) {
        best = c;
        *body_out = cand;
      }
    }
  }
  return best;
}

}  // namespace
}  // namespace ea

using namespace ea;

extern "C" int ea_exprog_simulate(const char* text, double link_gbs, double hbm_gbs, double* seconds) {
  if (!text || !seconds || !(link_gbs > 0) || !(hbm_gbs > 0)) return fail(EA_ERR_ARG, "ea_exprog_simulate: bad arguments");
  Prog p;
  int e = parse(text, &p);
  if (e) return e;
  std::vector<std::vector<int>> chosen;
  std::string why;
  bool found = false;
  memberships(p, [&](const std::vector<std::vector<int>>& mem) {
    std::string w;
    if (check(p, mem, &w)) {
      chosen = mem;
      found = true;
      return true;
    }
    if (why.empty()) why = w;
    return false;
  });
  if (!found) return fail(EA_ERR_ARG, "ea_exprog_simulate: the program is not valid: %s", why.c_str());
  const double t = simulate(p, chosen, link_gbs * 1e9, hbm_gbs * 1e9);
  if (t < 0) return fail(EA_ERR_ARG, "ea_exprog_simulate: the program stalls");
  *seconds = t;
  return ok();
}

extern "C" int ea_exprog_check(const char* text, int32_t* valid, char* why, int64_t why_cap) {
  if (!text || !valid) return fail(EA_ERR_ARG, "ea_exprog_check: NULL argument");
  Prog p;
  int e = parse(text, &p);
  if (e) return e;
  std::string first_why;
  bool ok_any = false;
  memberships(p, [&](const std::vector<std::vector<int>>& mem) {
    std::string w;
    if (check(p, mem, &w)) {
      ok_any = true;
      return true;
    }
    if (first_why.empty()) first_why = w;
    return false;
  });
  *valid = ok_any ? 1 : 0;
  if (why && why_cap > 0) {
    const std::string w = ok_any ? std::string() : first_why;
    const size_t n = std::min<size_t>(w.size(), (size_t)why_cap - 1);
    memcpy(why, w.data(), n);
    why[n] = 0;
  }
  return ok();
}

extern "C" int ea_exprog_naive(const char* text, char* out, int64_t cap, int64_t* len) {
  if (!text || !len) return fail(EA_ERR_ARG, "ea_exprog_naive: NULL argument");
  Prog p;
  int e = parse(text, &p);
  if (e) return e;
  std::vector<std::vector<int>> first;
  memberships(p, [&](const std::vector<std::vector<int>>& mem) {
    first = mem;
    return true;
  });
  std::string body;
  for (const FAct& f : naive_body(p, first)) body += render_act(p, f) + "\n";
  const std::string prog = p.decl_text + "\n" + body;
  *len = (int64_t)prog.size();
  if (!out || cap < (int64_t)prog.size() + 1)
    return fail(EA_ERR_CAPACITY, "ea_exprog_naive: %lld bytes needed", (long long)prog.size() + 1);
  memcpy(out, prog.data(), prog.size());
  out[prog.size()] = 0;
  return ok();
}

extern "C" int ea_exprog_synthesize(const char* text, double link_gbs, double hbm_gbs, int32_t iters, uint64_t seed,
                                    char* out, int64_t cap, int64_t* len, double* seconds) {
  if (!text || !len || !seconds || !(link_gbs > 0) || !(hbm_gbs > 0) || iters < 0)
    return fail(EA_ERR_ARG, "ea_exprog_synthesize: bad arguments");
  Prog p;
  int e = parse(text, &p);
  if (e) return e;
  std::vector<std::vector<int>> mem;
  std::vector<FAct> body;
  const double t = synthesize(p, link_gbs * 1e9, hbm_gbs * 1e9, iters, seed, &mem, &body);
  if (t < 0) return fail(EA_ERR_ARG, "ea_exprog_synthesize: no membership admits the naive program");
  std::string prog = render_decls(p, mem) + "\n";
  for (const FAct& f : body) prog += render_act(p, f) + "\n";
  *len = (int64_t)prog.size();
  *seconds = t;
  if (!out || cap < (int64_t)prog.size() + 1)
    return fail(EA_ERR_CAPACITY, "ea_exprog_synthesize: %lld bytes needed", (long long)prog.size() + 1);
  memcpy(out, prog.data(), prog.size());
  out[prog.size()] = 0;
  return ok();
}

extern "C" int ea_exprog_preamble(int32_t rank, const int32_t* prod_nblocks, const int64_t* prod_splits,
                                  int32_t n_prod, const int64_t* prod_block, const int32_t* prod_gpu,
                                  const int32_t* cons_nblocks, const int64_t* cons_splits, int32_t n_cons,
                                  const int64_t* cons_block, int32_t n_gpus, int64_t elem_bytes, char* out,
                                  int64_t cap, int64_t* len) {
  if (rank < 1 || rank > kMaxRank || !prod_nblocks || !prod_splits || !cons_nblocks || !cons_splits || !len ||
      n_prod < 1 || n_cons < 1 || n_gpus < 1 || !prod_block || !prod_gpu || !cons_block)
    return fail(EA_ERR_ARG, "ea_exprog_preamble: bad arguments");
  // partitions cover the GPUs (Section 5.2): one consumer specification per GPU
  if (n_cons != n_gpus)
    return fail(EA_ERR_ARG, "ea_exprog_preamble: %d consumer specifications for %d GPUs", n_cons, n_gpus);
  // the two tilings and their overlay (per dim: the union of split points)
  std::vector<std::vector<int64_t>> ps(rank), cs(rank), os(rank);
  for (int d = 0, pi = 0, ci = 0; d < rank; ++d) {
    if (prod_nblocks[d] < 1 || cons_nblocks[d] < 1) return fail(EA_ERR_ARG, "ea_exprog_preamble: dim %d has no blocks", d);
    ps[d].assign(prod_splits + pi, prod_splits + pi + prod_nblocks[d] + 1);
    cs[d].assign(cons_splits + ci, cons_splits + ci + cons_nblocks[d] + 1);
    pi += prod_nblocks[d] + 1;
    ci += cons_nblocks[d] + 1;
    for (const auto* v : {&ps[d], &cs[d]})
      for (size_t i = 0; i + 1 < v->size(); ++i)
        if ((*v)[i] >= (*v)[i + 1] || (*v)[0] != 0) return fail(EA_ERR_PARTITION, "ea_exprog_preamble: dim %d split points", d);
    if (ps[d].back() != cs[d].back()) return fail(EA_ERR_PARTITION, "ea_exprog_preamble: dim %d extents differ", d);
    std::set<int64_t> u(ps[d].begin(), ps[d].end());
    u.insert(cs[d].begin(), cs[d].end());
    os[d].assign(u.begin(), u.end());
  }
  int64_t n_pblocks = 1, n_cblocks = 1, n_atoms = 1;
  for (int d = 0; d < rank; ++d) {
    n_pblocks *= (int64_t)ps[d].size() - 1;
    n_cblocks *= (int64_t)cs[d].size() - 1;
    n_atoms *= (int64_t)os[d].size() - 1;
  }
  // block coordinates -> the overlay cells inside, in row-major order
  auto cells_of = [&](const std::vector<std::vector<int64_t>>& t, int64_t b) {
    int64_t rem = b;
    std::vector<std::pair<int64_t, int64_t>> rng(rank);  // overlay cell index range per dim
    for (int d = rank - 1; d >= 0; --d) {
      const int64_t n = (int64_t)t[d].size() - 1, c = rem % n;
      rem /= n;
      const int64_t lo = std::lower_bound(os[d].begin(), os[d].end(), t[d][c]) - os[d].begin();
      const int64_t hi = std::lower_bound(os[d].begin(), os[d].end(), t[d][c + 1]) - os[d].begin();
      rng[d] = {lo, hi};
    }
    std::vector<int64_t> out_cells;
    std::vector<int64_t> idx(rank);
    for (int d = 0; d < rank; ++d) idx[d] = rng[d].first;
    while (true) {
      int64_t a = 0;
      for (int d = 0; d < rank; ++d) a = a * ((int64_t)os[d].size() - 1) + idx[d];
      out_cells.push_back(a);
      int d = rank - 1;
      while (d >= 0 && ++idx[d] == rng[d].second) {
        idx[d] = rng[d].first;
        --d;
      }
      if (d < 0) break;
    }
    return out_cells;
  };
  auto atom_elems = [&](int64_t a) {
    int64_t n = 1, rem = a;
    for (int d = rank - 1; d >= 0; --d) {
      const int64_t k = (int64_t)os[d].size() - 1, c = rem % k;
      rem /= k;
      n *= os[d][c + 1] - os[d][c];
    }
    return n;
  };
  // copies of every atom: (copy letter, producer spec) in spec order
  const char* kCopy = "XYZWVUTSRQPONMLKJIHGFEDCBA";
  std::vector<std::vector<int>> copies((size_t)n_atoms);  // producer spec indices holding a copy
  std::vector<int> seen_per_block((size_t)n_pblocks, 0);
  std::vector<int> copy_of_spec((size_t)n_prod);
  for (int i = 0; i < n_prod; ++i) {
    if (prod_block[i] < 0 || prod_block[i] >= n_pblocks || prod_gpu[i] < 0 || prod_gpu[i] >= n_gpus)
      return fail(EA_ERR_ARG, "ea_exprog_preamble: producer spec %d: block or GPU out of range", i);
    copy_of_spec[(size_t)i] = seen_per_block[(size_t)prod_block[i]]++;
    if (copy_of_spec[(size_t)i] >= 26) return fail(EA_ERR_ARG, "ea_exprog_preamble: more than 26 copies of a block");
    for (int64_t a : cells_of(ps, prod_block[i])) copies[(size_t)a].push_back(i);
  }
  auto name = [&](int spec, int64_t atom) { return std::string(1, kCopy[copy_of_spec[(size_t)spec]]) + std::to_string(atom + 1); };
  std::string t = "GPUS: ";
  for (int gi = 0; gi < n_gpus; ++gi) t += (gi ? ", " : "") + std::to_string(gi);
  t += "\nPARTITIONS:";
  for (int j = 0; j < n_cons; ++j) t += " S" + std::to_string(j + 1) + " {size 1}";
  t += "\nIN: ";
  bool first = true;
  for (int i = 0; i < n_prod; ++i)
    for (int64_t a : cells_of(ps, prod_block[i])) {
      t += (first ? "" : "; ") + name(i, a) + " @ " + std::to_string(prod_gpu[i]);
      if (elem_bytes > 0) {
        char buf[64];
        snprintf(buf, sizeof(buf), " (size: %.9g GB)", (double)(atom_elems(a) * elem_bytes) / 1e9);
        t += buf;
      }
      first = false;
    }
  // the consumer specs reading each atom
  std::vector<std::vector<int>> readers((size_t)n_atoms);
  for (int j = 0; j < n_cons; ++j) {
    if (cons_block[j] < 0 || cons_block[j] >= n_cblocks)
      return fail(EA_ERR_ARG, "ea_exprog_preamble: consumer spec %d: block out of range", j);
    for (int64_t a : cells_of(cs, cons_block[j])) readers[(size_t)a].push_back(j);
  }
  t += "\nOUT: ";
  first = true;
  for (int64_t a = 0; a < n_atoms; ++a) {
    if (readers[(size_t)a].empty()) continue;
    if (copies[(size_t)a].empty()) return fail(EA_ERR_ARG, "ea_exprog_preamble: atom %lld has no copy", (long long)a + 1);
    std::string agg;
    for (int i : copies[(size_t)a]) agg += (agg.empty() ? "" : "+") + name(i, a);
    t += (first ? "" : "; ") + agg + " @ ";
    for (size_t k = 0; k < readers[(size_t)a].size(); ++k)
      t += (k ? ", S" : "S") + std::to_string(readers[(size_t)a][k] + 1);
    first = false;
  }
  t += "\n";
  *len = (int64_t)t.size();
  if (!out || cap < (int64_t)t.size() + 1) return fail(EA_ERR_CAPACITY, "ea_exprog_preamble: %lld bytes needed", (long long)t.size() + 1);
  memcpy(out, t.data(), t.size());
  out[t.size()] = 0;
  return ok();
}
