// Active-lane scheduler (host side): the paper's active-lane decoding
// algorithm (Section 3.3) around the three device calls.
//
// Each iteration the driver asks for a plan (the active lanes, depth-first
// in the lane tree with refine children before generate children), copies
// the lanes' token blocks out with al_sched_blocks, runs lane_attn_forward
// per prefix-state group, lmhead_confidence on the masked rows and
// select_unmask, and hands the updated blocks and lane statistics back to
// al_sched_commit, which writes them into the global sequence and applies
// the lane transitions:
// * a generate lane whose statistics say fork_ok forks at p = split
//   (eq. fork_operator): refine child (s, p), generate child
//   (s + p, min(B, L - s - p)) when s + p < L, both sharing a new
//   prefix-state group;
// * otherwise a lane whose region is filled completes; a completed
//   generate lane stops advancing when v = 0 or s + v >= L
//   ("Advancement control", cascading termination) and otherwise spawns a
//   successor generate lane at s + v in a new group.
// Write-back takes every lane's update region first, then lookahead drafts
// into positions still masked.  Model-call NFE counts one call per
// prefix-state group per iteration, plus one for the prompt (Section 3.4).
// Output reconstruction walks the tree: a forked lane emits its refine then
// its generate child, a lane that spawned emits [s, s+v) then its
// successor, a leaf emits its region up to its first mask (generate leaves
// also stop before EOS).
#include <stdint.h>

#include <algorithm>
#include <new>
#include <vector>

#include "../../include/asynclane.h"

namespace {

enum : int { KIND_NONE = 0, KIND_FORK = 1, KIND_SPAWN = 2 };

struct Lane {
  int role, s, b, parent, group, t, kind, v;
  bool done;
  std::vector<int> children;
};

}  // namespace

struct al_sched {
  int P, L, B, window, W, max_lanes, pad;
  std::vector<int32_t> tokens;
  std::vector<uint8_t> masked;
  std::vector<Lane> lanes;
  int next_group = 1, iterations = 0, nfe = 1, forks = 0, spawns = 0, stops = 0;
  std::vector<int> plan;  // lane ids of the last plan, in order

  void add(int parent, int role, int s, int b, int group) {
    Lane ln{role, s, b, parent, group, 0, KIND_NONE, 0, false, {}};
    lanes.push_back(ln);
    lanes[parent].children.push_back((int)lanes.size() - 1);
  }
};

extern "C" {

al_sched* al_sched_create(int P, int L_gen, int B, int window, int max_lanes, int pad_id) {
  if (P < 0 || L_gen < 1 || B < 1 || window < 0 || max_lanes < 1 || max_lanes > AL_MAX_LANES)
    return nullptr;
  al_sched* s = new (std::nothrow) al_sched();
  if (!s) return nullptr;
  s->P = P;
  s->L = L_gen;
  s->B = B;
  s->window = window;
  s->W = B + window;
  s->max_lanes = max_lanes;
  s->pad = pad_id;
  s->tokens.assign(L_gen, -1);
  s->masked.assign(L_gen, 1);
  s->lanes.push_back(Lane{AL_ROLE_GEN, 0, std::min(B, L_gen), -1, 0, 0, KIND_NONE, 0, false, {}});
  return s;
}

void al_sched_destroy(al_sched* s) { delete s; }

int al_sched_plan(al_sched* s, int32_t* lane_id, uint8_t* role, int32_t* start, int32_t* b_len,
                  int32_t* t_step, int32_t* group, int32_t* call_parent, int cap) {
  if (!s) return AL_ERR_NULL;
  s->plan.clear();
  std::vector<int> stack{0};
  while (!stack.empty() && (int)s->plan.size() < s->max_lanes) {
    const int id = stack.back();
    stack.pop_back();
    const Lane& ln = s->lanes[id];
    if (!ln.done) s->plan.push_back(id);
    for (auto it = ln.children.rbegin(); it != ln.children.rend(); ++it) stack.push_back(*it);
  }
  const int n = (int)s->plan.size();
  if (n > cap) return AL_ERR_SHAPE;
  if (n > 0 && (!lane_id || !role || !start || !b_len || !t_step || !group || !call_parent))
    return AL_ERR_NULL;
  for (int k = 0; k < n; ++k) {
    const Lane& ln = s->lanes[s->plan[k]];
    int cp = -1;
    // A generate child of a fork sees its refine sibling's block when the
    // sibling is evaluated in the same call (same prefix state).
    if (ln.role == AL_ROLE_GEN && ln.parent >= 0 && s->lanes[ln.parent].kind == KIND_FORK) {
      const int sib = s->lanes[ln.parent].children[0];
      for (int j = 0; j < k; ++j)
        if (s->plan[j] == sib && s->lanes[sib].group == ln.group) cp = j;
    }
    lane_id[k] = s->plan[k];
    role[k] = (uint8_t)ln.role;
    start[k] = ln.s;
    b_len[k] = ln.b;
    t_step[k] = ln.t + 1;  // the step count of eq. fork_condition includes this step
    group[k] = ln.group;
    call_parent[k] = cp;
  }
  return n;
}

int al_sched_blocks(const al_sched* s, int32_t* tokens, uint8_t* masked) {
  if (!s || (!s->plan.empty() && (!tokens || !masked))) return AL_ERR_NULL;
  const int W = s->W;
  for (size_t i = 0; i < s->plan.size(); ++i) {
    const int st = s->lanes[s->plan[i]].s;
    for (int a = 0; a < W; ++a) {
      const int pos = st + a;
      const bool in = pos < s->L;
      tokens[i * W + a] = in ? s->tokens[pos] : s->pad;  // past L: filled padding
      masked[i * W + a] = in ? s->masked[pos] : 0;
    }
  }
  return (int)s->plan.size();
}

int al_sched_commit(al_sched* s, const int32_t* tokens, const uint8_t* masked,
                    const int32_t* lane_stats) {
  if (!s) return AL_ERR_NULL;
  const int n = (int)s->plan.size();
  if (n > 0 && (!tokens || !masked || !lane_stats)) return AL_ERR_NULL;
  // The statistics come from select_unmask on the planned blocks; values
  // outside a lane's region are rejected before any state changes.
  for (int i = 0; i < n; ++i) {
    const int b = s->lanes[s->plan[i]].b;
    const int32_t* st = lane_stats + (size_t)i * AL_LANE_STATS;
    if (st[AL_STAT_SPLIT] < 0 || st[AL_STAT_SPLIT] > b || st[AL_STAT_FILLED] < 0 ||
        st[AL_STAT_FILLED] > b || st[AL_STAT_VALID] < 0 || st[AL_STAT_VALID] > b ||
        (st[AL_STAT_FORK] && st[AL_STAT_SPLIT] < 1))
      return AL_ERR_SHAPE;
  }
  const int W = s->W, L = s->L;
  for (int phase = 0; phase < 2; ++phase) {  // update regions, then window drafts
    for (int i = 0; i < n; ++i) {
      const Lane& ln = s->lanes[s->plan[i]];
      const int a0 = phase == 0 ? 0 : ln.b, a1 = phase == 0 ? ln.b : W;
      for (int a = a0; a < a1; ++a) {
        const int pos = ln.s + a;
        if (pos < L && s->masked[pos] && !masked[i * W + a]) {
          s->tokens[pos] = tokens[i * W + a];
          s->masked[pos] = 0;
        }
      }
    }
  }
  std::vector<int> groups;
  for (int i = 0; i < n; ++i) groups.push_back(s->lanes[s->plan[i]].group);
  std::sort(groups.begin(), groups.end());
  s->nfe += (int)(std::unique(groups.begin(), groups.end()) - groups.begin());
  s->iterations += 1;
  for (int i = 0; i < n; ++i) s->lanes[s->plan[i]].t += 1;
  for (int i = 0; i < n; ++i) {
    const int id = s->plan[i];
    const int32_t* st = lane_stats + (size_t)i * AL_LANE_STATS;
    const Lane ln = s->lanes[id];  // copy: add() may reallocate the vector
    if (ln.role == AL_ROLE_GEN && st[AL_STAT_FORK]) {
      const int p = st[AL_STAT_SPLIT];
      const int g = s->next_group++;
      s->add(id, AL_ROLE_REF, ln.s, p, g);
      if (ln.s + p < L) s->add(id, AL_ROLE_GEN, ln.s + p, std::min(s->B, L - ln.s - p), g);
      s->lanes[id].kind = KIND_FORK;
      s->lanes[id].done = true;
      s->forks += 1;
    } else if (st[AL_STAT_FILLED] == ln.b) {
      s->lanes[id].done = true;
      if (ln.role == AL_ROLE_GEN) {
        const int v = st[AL_STAT_VALID];
        if (v == 0 || ln.s + v >= L) {
          s->stops += 1;
        } else {
          const int g = s->next_group++;
          s->add(id, AL_ROLE_GEN, ln.s + v, std::min(s->B, L - ln.s - v), g);
          s->lanes[id].kind = KIND_SPAWN;
          s->lanes[id].v = v;
          s->spawns += 1;
        }
      }
    }
  }
  int active = 0;
  for (const Lane& ln : s->lanes) active += !ln.done;
  return active;
}

int al_sched_collect(const al_sched* s, int eos_id, int32_t* out, int cap) {
  if (!s || (cap > 0 && !out)) return AL_ERR_NULL;
  int n = 0;
  std::vector<int> stack{0};
  while (!stack.empty()) {
    const int id = stack.back();
    stack.pop_back();
    const Lane& ln = s->lanes[id];
    if (ln.kind == KIND_FORK) {
      for (auto it = ln.children.rbegin(); it != ln.children.rend(); ++it) stack.push_back(*it);
      continue;
    }
    const int len = ln.kind == KIND_SPAWN ? ln.v : ln.b;
    for (int a = 0; a < len; ++a) {
      const int pos = ln.s + a;
      if (ln.kind != KIND_SPAWN &&
          (s->masked[pos] || (ln.role == AL_ROLE_GEN && s->tokens[pos] == eos_id)))
        break;
      if (n >= cap) return AL_ERR_SHAPE;
      out[n++] = s->tokens[pos];
    }
    if (ln.kind == KIND_SPAWN) stack.push_back(ln.children[0]);
  }
  return n;
}

int al_sched_counters(const al_sched* s, int32_t* out) {
  if (!s || !out) return AL_ERR_NULL;
  out[0] = s->iterations;
  out[1] = s->nfe;
  out[2] = s->forks;
  out[3] = s->spawns;
  out[4] = s->stops;
  out[5] = (int32_t)s->lanes.size();
  return AL_OK;
}

int al_sched_tree(const al_sched* s, uint8_t* role, int32_t* start, int32_t* length,
                  int32_t* parent, int32_t* kind, int32_t* v, int cap) {
  if (!s) return AL_ERR_NULL;
  const int n = (int)s->lanes.size();
  if (n > cap) return AL_ERR_SHAPE;
  if (!role || !start || !length || !parent || !kind || !v) return AL_ERR_NULL;
  for (int i = 0; i < n; ++i) {
    const Lane& ln = s->lanes[i];
    role[i] = (uint8_t)ln.role;
    start[i] = ln.s;
    length[i] = ln.b;
    parent[i] = ln.parent;
    kind[i] = ln.kind;
    v[i] = ln.kind == KIND_SPAWN ? ln.v : -1;
  }
  return n;
}

int al_sched_state(const al_sched* s, int32_t* tokens, uint8_t* masked) {
  if (!s || !tokens || !masked) return AL_ERR_NULL;
  std::copy(s->tokens.begin(), s->tokens.end(), tokens);
  std::copy(s->masked.begin(), s->masked.end(), masked);
  return s->L;
}

}  // extern "C"
