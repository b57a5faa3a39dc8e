// Host-side bidirectional KV block manager and the priority-based packing
// scheduler (Sec. 5.2 Block Management; Sec. 4.2 Alg. 1 and adaptive batch
// sizing). Pure C++: it decides where tokens go and what must move; the
// kernels move the bytes.
//
// Blocks have 16 slots. A block holds at most one RT owner, filling slots from
// the left, and one BE owner, filling them from the right (Sec. 5.1). Each
// owner treats the block as its own 16 positions (entry e of a request's table
// holds its positions [16 e, 16 e + 16)). The manager keeps, per block, how
// many of each owner's tokens are still in it:
//   RT: slots [0, rt_n)        BE: slots [16 - be_n, 16)
// and, per request entry, how many of the entry's leading positions are on
// the GPU; positions of the entry beyond that were checkpointed to CPU memory.
//
// Growth of a request by one token at position p (entry e = p / 16):
//   * a new entry takes a block: a free block if any, else the block with the
//     most empty slots among those without an owner of the request's class
//     (FindBlock; for RT this is FindPreemptBlock, which takes BE blocks);
//   * the token's slot is free: it is placed;
//   * the slot holds the peer's token and the writer is RT: the peer's token
//     is checkpointed (a victim, gathered before the write) and the block is
//     marked preempted (lazy checkpointing);
//   * the slot holds the peer's token and the writer is BE: BE never
//     overwrites RT; its entry moves to another block (a relocation: device
//     moves of the entry's tokens), where the token is placed.
// Restoring a request with checkpointed tokens (before it runs again): each
// such entry is rebuilt where the checkpointed slots are free, in place when
// its block has room, else in another block with its surviving tokens moved.
#include "bros_attn.h"
#include "bros_error.h"

#include <algorithm>
#include <cstdint>
#include <iterator>
#include <limits>
#include <cstdio>
#include <set>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

using bros::fail;

namespace {

constexpr int kBS = 16;

struct Block {
  int32_t rt = -1, be = -1;     // owners (request ids)
  int32_t rt_e = 0, be_e = 0;   // the owners' table entries mapped here
  int32_t rt_n = 0, be_n = 0;   // their tokens present in the block
  bool preempted = false;
  // Which block list holds the block (at most one: free, RT-open or BE-open)
  // and under which count of empty slots, so that a list update touches only
  // the list the block is in.
  int8_t listed = 0;   // kListedRt | kListedBe | kListedFree
  int8_t key = 0;
  int empty() const { return kBS - rt_n - be_n; }
};
constexpr int8_t kListedRt = 1, kListedBe = 2, kListedFree = 4;

struct Request {
  int32_t cls = BROS_RT;
  int32_t ctx = 0;                  // tokens the request holds (on the GPU or checkpointed)
  std::vector<int32_t> table;       // block of each entry
  std::vector<int32_t> on_gpu;      // leading positions of each entry present on the GPU
  int32_t missing = 0;              // tokens checkpointed to CPU memory (kept equal to the sum below)
  int dir() const { return cls == BROS_BE ? -1 : 1; }
  int32_t count(size_t e) const { return std::min<int32_t>(kBS, ctx - (int32_t)e * kBS); }
  int32_t checkpointed() const { return missing; }
  int32_t checkpointed_by_entries() const {
    int32_t n = 0;
    for (size_t e = 0; e < table.size(); ++e) n += count(e) - on_gpu[e];
    return n;
  }
};

int slot_of(int dir, int off) { return dir > 0 ? off : kBS - 1 - off; }

struct Plan {
  std::vector<int32_t> victims;   // 4 per token: request, position, block, slot
  std::vector<int32_t> move_src, move_dst;
  std::vector<int32_t> restore_pos, restore_dst;
  std::vector<std::pair<int32_t, int32_t>> written;   // (position, slot id) of each new token
};

class Manager {
 public:
  explicit Manager(int32_t n) : blocks_(n) {
    for (int32_t b = 0; b < n; ++b) {
      free_.insert(b);
      blocks_[b].listed = kListedFree;
    }
  }

  int32_t num_blocks() const { return (int32_t)blocks_.size(); }
  int32_t free_blocks() const { return (int32_t)free_.size(); }
  bool has(int32_t id) const { return reqs_.count(id) != 0; }
  const Request& req(int32_t id) const { return reqs_.at(id); }
  const Block& block(int32_t b) const { return blocks_[b]; }

  void add(int32_t id, int32_t cls) { reqs_[id].cls = cls; }

  // Blocks a request of class `cls` could take for a new entry: free ones,
  // and ones without an owner of that class (counted once each).
  int32_t available_for(int32_t cls) const { return free_blocks() + open_for(cls); }

  // Non-free blocks a new entry of class cls may take: for RT every block
  // without an RT owner (preempting its BE owner), for BE every block without
  // a BE owner that still has an empty slot.
  int32_t open_for(int32_t cls) const {
    if (cls == BROS_RT) return (int32_t)rt_open_.size();
    // be_open_ is ordered by empty slots, most first: count up to the first full one
    auto full = be_open_.lower_bound({0, std::numeric_limits<int32_t>::min()});
    return (int32_t)std::distance(be_open_.begin(), full);
  }

  // New entries (blocks) that growing `id` by n tokens takes, not counting
  // relocations (a BE entry that meets an RT token moves, taking one more).
  int32_t entries_needed(int32_t id, int32_t n) const {
    const Request& r = reqs_.at(id);
    const int32_t have = (int32_t)r.table.size();
    const int32_t need = (r.ctx + n + kBS - 1) / kBS;
    return std::max(0, need - have);
  }

  // One new token for request id; false if no block can be found (the
  // manager is then unchanged for this token).
  bool grow_one(int32_t id, Plan& plan) {
    Request& r = reqs_.at(id);
    const int32_t p = r.ctx;
    const int32_t e = p / kBS, off = p % kBS;
    if ((size_t)e == r.table.size()) {
      const int32_t b = take_block(r.cls, -1, 1);
      if (b < 0) return false;
      attach(id, r, e, b);
    }
    int32_t b = r.table[e];
    const int s = slot_of(r.dir(), off);
    Block& blk = blocks_[b];
    unlist(b);
    const bool peer_holds = r.cls == BROS_RT ? (blk.be >= 0 && s >= kBS - blk.be_n) : (blk.rt >= 0 && s < blk.rt_n);
    if (peer_holds) {
      if (r.cls == BROS_RT) {
        // lazy checkpointing: the BE peer's innermost token goes to CPU memory
        Request& peer = reqs_.at(blk.be);
        const int32_t pe = blk.be_e;
        const int32_t ppos = pe * kBS + (kBS - 1 - s);
        plan.victims.insert(plan.victims.end(), {blk.be, ppos, b, s});
        blk.be_n -= 1;
        peer.on_gpu[pe] -= 1;
        peer.missing += 1;
        blk.preempted = true;
      } else {
        // BE never overwrites RT: its entry moves to another block
        refresh(b);
        const int32_t nb = take_block(r.cls, b, r.on_gpu[e] + 1);
        if (nb < 0) return false;
        relocate(id, r, e, nb, plan);
        b = nb;
        unlist(b);
      }
    }
    Block& dst = blocks_[b];
    if (r.cls == BROS_RT) dst.rt_n += 1; else dst.be_n += 1;
    r.on_gpu[e] = off + 1;
    r.ctx += 1;
    plan.written.emplace_back(p, b * kBS + s);
    refresh(b);
    return true;
  }

  // Checkpointed tokens of `id` back to the GPU (before it runs again).
  bool restore(int32_t id, Plan& plan) {
    Request& r = reqs_.at(id);
    if (r.missing == 0) return true;
    for (size_t e = 0; e < r.table.size(); ++e) {
      const int32_t cnt = r.count(e);
      if (r.on_gpu[e] >= cnt) continue;
      int32_t b = r.table[e];
      Block& blk = blocks_[b];
      // room in place: none of the entry's missing slots is held by the peer
      bool in_place = true;
      for (int32_t off = r.on_gpu[e]; off < cnt; ++off) {
        const int s = slot_of(r.dir(), off);
        if (r.cls == BROS_BE ? (blk.rt >= 0 && s < blk.rt_n) : (blk.be >= 0 && s >= kBS - blk.be_n)) in_place = false;
      }
      if (!in_place) {
        const int32_t nb = take_block(r.cls, b, cnt);
        if (nb < 0) return false;
        relocate(id, r, (int32_t)e, nb, plan);
        b = nb;
      }
      unlist(b);
      Block& dst = blocks_[b];
      for (int32_t off = r.on_gpu[e]; off < cnt; ++off) {
        plan.restore_pos.push_back((int32_t)e * kBS + off);
        plan.restore_dst.push_back(b * kBS + slot_of(r.dir(), off));
      }
      if (r.cls == BROS_RT) dst.rt_n += cnt - r.on_gpu[e]; else dst.be_n += cnt - r.on_gpu[e];
      r.missing -= cnt - r.on_gpu[e];
      r.on_gpu[e] = cnt;
      refresh(b);
    }
    return true;
  }

  void release(int32_t id) {
    Request& r = reqs_.at(id);
    for (size_t e = 0; e < r.table.size(); ++e) detach(id, r.table[e]);
    reqs_.erase(id);
  }

  // Every internal invariant; returns a description of the first broken one
  // (empty when all hold).
  std::string validate() const {
    char buf[256];
    for (const auto& kv : reqs_) {
      const int32_t id = kv.first;
      const Request& r = kv.second;
      if (r.table.size() != r.on_gpu.size()) return "table/on_gpu size mismatch";
      if ((int32_t)r.table.size() != (r.ctx + kBS - 1) / kBS) {
        snprintf(buf, sizeof buf, "request %d: %zu entries for ctx %d", id, r.table.size(), r.ctx);
        return buf;
      }
      for (size_t e = 0; e < r.table.size(); ++e) {
        const Block& b = blocks_[r.table[e]];
        const bool rt = r.cls == BROS_RT;
        if ((rt ? b.rt : b.be) != id || (rt ? b.rt_e : b.be_e) != (int32_t)e || (rt ? b.rt_n : b.be_n) != r.on_gpu[e]) {
          snprintf(buf, sizeof buf, "request %d entry %zu: block %d has owner %d entry %d count %d (expected count %d)",
                   id, e, r.table[e], rt ? b.rt : b.be, rt ? b.rt_e : b.be_e, rt ? b.rt_n : b.be_n, r.on_gpu[e]);
          return buf;
        }
        if (r.on_gpu[e] < 0 || r.on_gpu[e] > r.count(e)) return "on_gpu out of range";
      }
      if (r.missing != r.checkpointed_by_entries()) {
        snprintf(buf, sizeof buf, "request %d: %d tokens counted as checkpointed, %d by entries", id, r.missing,
                 r.checkpointed_by_entries());
        return buf;
      }
    }
    for (int32_t i = 0; i < num_blocks(); ++i) {
      const Block& b = blocks_[i];
      if (b.rt_n + b.be_n > kBS || b.rt_n < 0 || b.be_n < 0) {
        snprintf(buf, sizeof buf, "block %d: counts %d + %d", i, b.rt_n, b.be_n);
        return buf;
      }
      if (b.rt >= 0 && (!reqs_.count(b.rt) || reqs_.at(b.rt).table[b.rt_e] != i)) {
        snprintf(buf, sizeof buf, "block %d: RT owner %d does not map entry %d here", i, b.rt, b.rt_e);
        return buf;
      }
      if (b.be >= 0 && (!reqs_.count(b.be) || reqs_.at(b.be).table[b.be_e] != i)) {
        snprintf(buf, sizeof buf, "block %d: BE owner %d does not map entry %d here", i, b.be, b.be_e);
        return buf;
      }
      const bool is_free = free_.count(i) != 0;
      const bool in_rt = rt_open_.count({-b.empty(), i}) != 0, in_be = be_open_.count({-b.empty(), i}) != 0;
      if (is_free != (b.rt < 0 && b.be < 0) || in_rt != (b.rt < 0 && b.be >= 0) || in_be != (b.be < 0 && b.rt >= 0)) {
        snprintf(buf, sizeof buf, "block %d: listed free %d rt-open %d be-open %d with owners %d/%d", i, is_free, in_rt,
                 in_be, b.rt, b.be);
        return buf;
      }
    }
    if (free_.size() + rt_open_.size() + be_open_.size() > blocks_.size()) return "stale entries in the block lists";
    return "";
  }

  std::vector<std::pair<int32_t, std::pair<int32_t, int32_t>>> preemption_table() const {
    std::vector<std::pair<int32_t, std::pair<int32_t, int32_t>>> out;
    for (int32_t b = 0; b < num_blocks(); ++b)
      if (blocks_[b].preempted) out.push_back({b, {blocks_[b].rt, blocks_[b].be}});
    return out;
  }

 private:
  // Sets of blocks that a new entry of one class may take besides free ones,
  // ordered by empty slots (most first): RT may take BE-only blocks, BE may
  // take RT-only blocks.
  using OpenSet = std::set<std::pair<int, int32_t>>;   // (-empty, block)

  // A block for a new or moving entry: a free block, else the open block
  // with the most empty slots. A BE entry needs `need` empty slots at the
  // right end (the RT owner fills from the left, so any `need` empty slots
  // are the right ones); RT takes any BE block (FindPreemptBlock).
  int32_t take_block(int32_t cls, int32_t exclude, int32_t need) {
    if (!free_.empty()) {
      const int32_t b = *free_.begin();
      free_.erase(free_.begin());
      blocks_[b].listed = 0;
      return b;
    }
    OpenSet& open = cls == BROS_RT ? rt_open_ : be_open_;
    for (auto it = open.begin(); it != open.end(); ++it) {
      if (cls == BROS_BE && -it->first < need) break;   // sorted by empty slots, most first
      if (it->second == exclude) continue;
      const int32_t b = it->second;
      open.erase(it);
      blocks_[b].listed = 0;
      return b;
    }
    return -1;
  }

  void attach(int32_t id, Request& r, int32_t e, int32_t b) {
    Block& blk = blocks_[b];
    unlist(b);
    if (r.cls == BROS_RT) { blk.rt = id; blk.rt_e = e; blk.rt_n = 0; }
    else { blk.be = id; blk.be_e = e; blk.be_n = 0; }
    if ((size_t)e == r.table.size()) { r.table.push_back(b); r.on_gpu.push_back(0); }
    else r.table[e] = b;
    refresh(b);
  }

  void detach(int32_t id, int32_t b) {
    Block& blk = blocks_[b];
    unlist(b);
    if (blk.rt == id) { blk.rt = -1; blk.rt_n = 0; }
    if (blk.be == id) { blk.be = -1; blk.be_n = 0; }
    if (blk.rt < 0 || blk.be < 0) blk.preempted = false;
    refresh(b);
  }

  // Entry e of request id moves to block nb: its tokens present on the GPU
  // are moved slot for slot; the old block loses this owner.
  void relocate(int32_t id, Request& r, int32_t e, int32_t nb, Plan& plan) {
    const int32_t ob = r.table[e];
    for (int32_t off = 0; off < r.on_gpu[e]; ++off) {
      const int s = slot_of(r.dir(), off);
      plan.move_src.push_back(ob * kBS + s);
      plan.move_dst.push_back(nb * kBS + s);
    }
    const int32_t keep = r.on_gpu[e];
    detach(id, ob);
    attach(id, r, e, nb);
    unlist(nb);
    Block& dst = blocks_[nb];
    if (r.cls == BROS_RT) dst.rt_n = keep; else dst.be_n = keep;
    refresh(nb);
  }

  void unlist(int32_t b) {
    Block& bl = blocks_[b];
    if (bl.listed & kListedRt) rt_open_.erase({-bl.key, b});
    if (bl.listed & kListedBe) be_open_.erase({-bl.key, b});
    if (bl.listed & kListedFree) free_.erase(b);
    bl.listed = 0;
  }

  void refresh(int32_t b) {
    const Block& blk = blocks_[b];
    const int8_t want = (blk.rt < 0 && blk.be < 0) ? kListedFree
                        : (blk.rt < 0 ? kListedRt : 0) | (blk.be < 0 ? kListedBe : 0);
    const int8_t key = (int8_t)blk.empty();
    if (blk.listed == want && (want == 0 || want == kListedFree || blk.key == key)) return;   // already so
    unlist(b);
    Block& bl = blocks_[b];
    bl.listed = want;
    bl.key = key;
    if (want == kListedFree) {
      free_.insert(b);
      return;
    }
    if (want & kListedRt) rt_open_.insert({-key, b});
    if (want & kListedBe) be_open_.insert({-key, b});
  }

  std::vector<Block> blocks_;
  std::set<int32_t> free_;
  OpenSet rt_open_, be_open_;
  std::unordered_map<int32_t, Request> reqs_;
};

Manager* as_mgr(void* m) { return static_cast<Manager*>(m); }

int copy_plan(const Plan& p, bros_mgr_plan* out) {
  if (out == nullptr) return BROS_OK;
  out->num_victims = (int32_t)(p.victims.size() / 4);
  out->num_moves = (int32_t)p.move_src.size();
  out->num_restores = (int32_t)p.restore_pos.size();
  out->num_written = (int32_t)p.written.size();
  if (out->num_victims > out->victims_cap || out->num_moves > out->moves_cap ||
      out->num_restores > out->restores_cap || out->num_written > out->written_cap)
    return fail(BROS_E_SHAPE, "plan buffers too small: %d victims, %d moves, %d restores, %d written",
                out->num_victims, out->num_moves, out->num_restores, out->num_written);
  std::copy(p.victims.begin(), p.victims.end(), out->victims);
  std::copy(p.move_src.begin(), p.move_src.end(), out->move_src);
  std::copy(p.move_dst.begin(), p.move_dst.end(), out->move_dst);
  std::copy(p.restore_pos.begin(), p.restore_pos.end(), out->restore_pos);
  std::copy(p.restore_dst.begin(), p.restore_dst.end(), out->restore_dst);
  for (size_t i = 0; i < p.written.size(); ++i) {
    out->written_pos[i] = p.written[i].first;
    out->written_slot[i] = p.written[i].second;
  }
  return BROS_OK;
}

}  // namespace

extern "C" {

void* bros_mgr_create(int32_t num_blocks) {
  if (num_blocks <= 0) {
    fail(BROS_E_SHAPE, "bros_mgr_create: num_blocks %d must be positive", num_blocks);
    return nullptr;
  }
  return new Manager(num_blocks);
}

void bros_mgr_destroy(void* mgr) { delete as_mgr(mgr); }

int bros_mgr_add_request(void* mgr, int32_t req, int32_t cls) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_add_request: mgr is NULL");
  if (cls != BROS_RT && cls != BROS_BE) return fail(BROS_E_SHAPE, "bros_mgr_add_request: class %d", cls);
  if (as_mgr(mgr)->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_add_request: request %d exists", req);
  as_mgr(mgr)->add(req, cls);
  return bros::ok();
}

int bros_mgr_release(void* mgr, int32_t req) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_release: mgr is NULL");
  if (!as_mgr(mgr)->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_release: no request %d", req);
  as_mgr(mgr)->release(req);
  return bros::ok();
}

int bros_mgr_grow(void* mgr, int32_t req, int32_t n_new, bros_mgr_plan* plan) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_grow: mgr is NULL");
  Manager* m = as_mgr(mgr);
  if (!m->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_grow: no request %d", req);
  if (n_new < 0) return fail(BROS_E_SHAPE, "bros_mgr_grow: n_new %d", n_new);
  if (m->req(req).checkpointed() > 0)
    return fail(BROS_E_TABLE, "bros_mgr_grow: request %d has checkpointed tokens; restore it first", req);
  Plan p;
  for (int32_t i = 0; i < n_new; ++i)
    if (!m->grow_one(req, p)) {
      copy_plan(p, plan);
      return fail(BROS_E_NOMEM, "bros_mgr_grow: no block for request %d after %d of %d tokens", req, i, n_new);
    }
  return copy_plan(p, plan);
}

int bros_mgr_grow_batch(void* mgr, const int32_t* reqs, const int32_t* n_new, int32_t n, int32_t restore_first,
                        bros_mgr_plan* plan, int32_t* ends, int32_t* status) {
  const char* fn = "bros_mgr_grow_batch";
  if (!mgr) return fail(BROS_E_NULL, "%s: mgr is NULL", fn);
  if (n < 0) return fail(BROS_E_SHAPE, "%s: n %d", fn, n);
  if (n > 0 && (!reqs || !n_new || !ends || !status)) return fail(BROS_E_NULL, "%s: NULL list", fn);
  Manager* m = as_mgr(mgr);
  for (int32_t i = 0; i < n; ++i) {   // arguments first: nothing changes for a bad call
    if (!m->has(reqs[i])) return fail(BROS_E_SHAPE, "%s: no request %d (index %d)", fn, reqs[i], i);
    if (n_new[i] < 0) return fail(BROS_E_SHAPE, "%s: n_new %d (index %d)", fn, n_new[i], i);
  }
  Plan p;
  int first_err = BROS_OK, first_idx = -1;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t req = reqs[i];
    int st = BROS_OK;
    if (m->req(req).checkpointed() > 0) {
      if (!restore_first) st = BROS_E_TABLE;
      else if (!m->restore(req, p)) st = BROS_E_NOMEM;
    }
    for (int32_t k = 0; st == BROS_OK && k < n_new[i]; ++k)
      if (!m->grow_one(req, p)) st = BROS_E_NOMEM;
    status[i] = st;
    if (st != BROS_OK && first_err == BROS_OK) {
      first_err = st;
      first_idx = i;
    }
    ends[4 * i + 0] = (int32_t)(p.victims.size() / 4);
    ends[4 * i + 1] = (int32_t)p.move_src.size();
    ends[4 * i + 2] = (int32_t)p.restore_pos.size();
    ends[4 * i + 3] = (int32_t)p.written.size();
  }
  const int cst = copy_plan(p, plan);
  if (cst != BROS_OK) return cst;
  if (first_err != BROS_OK)
    return fail(first_err, "%s: request %d (index %d) %s; the other requests' results are in the plan", fn,
                reqs[first_idx], first_idx,
                first_err == BROS_E_NOMEM ? "found no block" : "has checkpointed tokens and restore_first is 0");
  return bros::ok();
}

int32_t bros_mgr_plan_bound(void* mgr, const int32_t* reqs, const int32_t* n_new, int32_t n) {
  if (!mgr || n < 0 || (n > 0 && (!reqs || !n_new))) return -1;
  Manager* m = as_mgr(mgr);
  int64_t cap = 64;
  for (int32_t i = 0; i < n; ++i) {
    if (!m->has(reqs[i]) || n_new[i] < 0) return -1;
    // a new token victimises at most one peer token and a relocation moves at
    // most 15; a restore moves or restores at most the request's tokens
    cap += 16 * (int64_t)n_new[i] + m->req(reqs[i]).ctx + 16;
  }
  return cap > 0x7fffffff ? -1 : (int32_t)cap;
}

int bros_mgr_restore(void* mgr, int32_t req, bros_mgr_plan* plan) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_restore: mgr is NULL");
  Manager* m = as_mgr(mgr);
  if (!m->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_restore: no request %d", req);
  Plan p;
  if (!m->restore(req, p)) {
    copy_plan(p, plan);
    return fail(BROS_E_NOMEM, "bros_mgr_restore: no block to restore request %d", req);
  }
  return copy_plan(p, plan);
}

int bros_mgr_query(void* mgr, int32_t req, int32_t* ctx, int32_t* num_entries, int32_t* checkpointed) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_query: mgr is NULL");
  Manager* m = as_mgr(mgr);
  if (!m->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_query: no request %d", req);
  const Request& r = m->req(req);
  if (ctx) *ctx = r.ctx;
  if (num_entries) *num_entries = (int32_t)r.table.size();
  if (checkpointed) *checkpointed = r.checkpointed();
  return bros::ok();
}

int bros_mgr_table(void* mgr, int32_t req, int32_t* out, int32_t cap) {
  if (!mgr || !out) return fail(BROS_E_NULL, "bros_mgr_table: NULL argument");
  Manager* m = as_mgr(mgr);
  if (!m->has(req)) return fail(BROS_E_SHAPE, "bros_mgr_table: no request %d", req);
  const Request& r = m->req(req);
  if ((int32_t)r.table.size() > cap) return fail(BROS_E_SHAPE, "bros_mgr_table: %zu entries > cap %d", r.table.size(), cap);
  std::copy(r.table.begin(), r.table.end(), out);
  return bros::ok();
}

int bros_mgr_validate(void* mgr) {
  if (!mgr) return fail(BROS_E_NULL, "bros_mgr_validate: mgr is NULL");
  const std::string why = as_mgr(mgr)->validate();
  if (!why.empty()) return fail(BROS_E_TABLE, "bros_mgr_validate: %s", why.c_str());
  return bros::ok();
}

int32_t bros_mgr_free_blocks(void* mgr) { return mgr ? as_mgr(mgr)->free_blocks() : -1; }

int32_t bros_mgr_available(void* mgr, int32_t cls) { return mgr ? as_mgr(mgr)->available_for(cls) : -1; }

int32_t bros_mgr_entries_needed(void* mgr, int32_t req, int32_t n_new) {
  if (!mgr || !as_mgr(mgr)->has(req)) return -1;
  return as_mgr(mgr)->entries_needed(req, n_new);
}

int32_t bros_mgr_preemption_table(void* mgr, int32_t* out, int32_t cap) {
  if (!mgr) return -1;
  const auto t = as_mgr(mgr)->preemption_table();
  for (int32_t i = 0; i < (int32_t)t.size() && i < cap; ++i) {
    out[3 * i] = t[i].first;
    out[3 * i + 1] = t[i].second.first;
    out[3 * i + 2] = t[i].second.second;
  }
  return (int32_t)t.size();
}

// --- Alg. 1 ------------------------------------------------------------------

// C(batch) of Sec. 4.1 kept as running sums, so adding or removing one
// request costs O(1): per phase a0 * Ln + a1 * X + b over the phase's
// requests (X = Ln * La, the paper's form, or the sum of n_i * a_i); a phase
// with no request costs nothing.
struct CostSums {
  double ln[2] = {0, 0}, la[2] = {0, 0}, pairs[2] = {0, 0};
  int cnt[2] = {0, 0};
  void add(const bros_sched_req* r, int sign) {
    const int ph = r->prefill ? 0 : 1;
    ln[ph] += sign * (double)r->n_new;
    la[ph] += sign * (double)r->ctx_after;
    pairs[ph] += sign * (double)r->n_new * r->ctx_after;
    cnt[ph] += sign;
  }
  double cost(const bros_cost_model* cm) const {
    double t = 0;
    for (int ph = 0; ph < 2; ++ph) {
      if (!cnt[ph]) continue;
      const double* a = cm->coef[ph];
      const double x = cm->per_request ? pairs[ph] : ln[ph] * la[ph];
      t += a[0] * ln[ph] + a[1] * x + a[2];
    }
    return t;
  }
};

}  // extern "C"

namespace {

// Alg. 1 over RT requests already in ascending order of remaining time (qrt)
// and BE requests in ascending order of checkpointed slots (qbe). The RT loop
// reads at most batch_size entries of qrt and the BE loop at most
// 2 batch_size + 1 of qbe (each BE step adds one request to the batch or
// replaces one RT request, else stops), so callers may pass only those
// prefixes.
int schedule_ordered(Manager* m, const std::vector<const bros_sched_req*>& qrt,
                     const std::vector<const bros_sched_req*>& qbe, int32_t batch_size, const bros_cost_model* cost,
                     int32_t* rt_ready, int32_t* n_rt_ready, int32_t* be_ready, int32_t* n_be_ready,
                     int32_t* over_budget) {
  const double t_res = qrt.empty() ? std::numeric_limits<double>::infinity() : qrt.front()->remaining_us;
  // Blocks the batch may still take (FindPreemptBlock / FindBlock): free ones
  // first, then RT may take blocks without an RT owner (preempting BE) and BE
  // blocks without a BE owner that have an empty slot.
  int32_t free_left = m->free_blocks();
  int32_t open_left[2] = {m->open_for(BROS_RT), m->open_for(BROS_BE)};
  auto need_of = [&](const bros_sched_req* r) -> int32_t {
    if (!m->has(r->id)) return (r->ctx_after + kBS - 1) / kBS;
    const Request& q = m->req(r->id);
    int32_t moved = 0;   // entries with checkpointed tokens may move on restore
    if (q.missing)
      for (size_t e = 0; e < q.table.size(); ++e) moved += q.on_gpu[e] < q.count(e);
    return m->entries_needed(r->id, r->n_new) + moved;
  };
  auto take = [&](int32_t need, int32_t cls, bool commit) -> bool {
    const int32_t from_free = std::min(need, free_left);
    const int32_t rest = need - from_free;
    if (rest > open_left[cls]) return false;
    if (commit) {
      free_left -= from_free;
      open_left[cls] -= rest;
    }
    return true;
  };
  std::vector<const bros_sched_req*> ready_rt, ready_be;
  CostSums sums;   // the requests in ready_rt and ready_be
  *over_budget = 0;
  size_t head = 0;
  while (head < qrt.size()) {
    const bros_sched_req* r = qrt[head];
    if ((int32_t)ready_rt.size() == batch_size) break;
    const int32_t need = need_of(r);
    if (!take(need, BROS_RT, false)) break;             // FindPreemptBlock fails
    CostSums cand = sums;
    cand.add(r, 1);
    if (cand.cost(cost) > t_res) {
      *over_budget = 1;
      break;
    }
    ++head;
    take(need, BROS_RT, true);
    ready_rt.push_back(r);
    sums = cand;
  }
  size_t bhead = 0;
  while (bhead < qbe.size()) {
    const bros_sched_req* r = qbe[bhead];
    const int32_t need = need_of(r);
    if (!take(need, BROS_BE, false)) break;             // FindBlock fails
    auto fits = [&](const CostSums& base, size_t n_ready) {
      CostSums cand = base;
      cand.add(r, 1);
      return (int32_t)(n_ready + 1) <= batch_size && cand.cost(cost) <= t_res;
    };
    if (fits(sums, ready_rt.size() + ready_be.size())) {
      ready_be.push_back(r);
      sums.add(r, 1);
    } else {
      if (ready_rt.empty()) break;
      const bros_sched_req* back = ready_rt.back();     // the least urgent RT request
      CostSums without = sums;
      without.add(back, -1);
      if (fits(without, ready_rt.size() - 1 + ready_be.size())) {
        ready_rt.pop_back();                            // `back` returns to the RT queue
        ready_be.push_back(r);
        sums = without;
        sums.add(r, 1);
      } else {
        break;
      }
    }
    take(need, BROS_BE, true);
    ++bhead;
  }
  for (size_t i = 0; i < ready_rt.size(); ++i) rt_ready[i] = ready_rt[i]->id;
  for (size_t i = 0; i < ready_be.size(); ++i) be_ready[i] = ready_be[i]->id;
  *n_rt_ready = (int32_t)ready_rt.size();
  *n_be_ready = (int32_t)ready_be.size();
  return bros::ok();
}

// The first k requests of q (pointers) in ascending key order, ties by
// position: a partial sort, O(n log k).
template <typename Key>
void first_k_sorted(std::vector<const bros_sched_req*>& q, size_t k, Key key) {
  k = std::min(k, q.size());
  const bros_sched_req* base = q.empty() ? nullptr : q.front();
  auto less = [&](const bros_sched_req* a, const bros_sched_req* b) {
    const auto ka = key(a), kb = key(b);
    return ka < kb || (ka == kb && a < b);   // entries point into one array: address order is position order
  };
  (void)base;
  std::partial_sort(q.begin(), q.begin() + k, q.end(), less);
  q.resize(k);
}

}  // namespace

extern "C" {

int bros_schedule(void* mgr, const bros_sched_req* rt, int32_t n_rt, const bros_sched_req* be, int32_t n_be,
                  int32_t batch_size, const bros_cost_model* cost, int32_t* rt_ready, int32_t* n_rt_ready,
                  int32_t* be_ready, int32_t* n_be_ready, int32_t* over_budget) {
  const char* fn = "bros_schedule";
  if (!mgr || !cost || !rt_ready || !n_rt_ready || !be_ready || !n_be_ready || !over_budget)
    return fail(BROS_E_NULL, "%s: NULL argument", fn);
  if ((n_rt > 0 && !rt) || (n_be > 0 && !be) || n_rt < 0 || n_be < 0 || batch_size < 0)
    return fail(BROS_E_SHAPE, "%s: bad queue arguments", fn);
  // RT queue in ascending remaining time; T_res_min is the most urgent's.
  std::vector<const bros_sched_req*> qrt, qbe;
  for (int32_t i = 0; i < n_rt; ++i) qrt.push_back(&rt[i]);
  for (int32_t i = 0; i < n_be; ++i) qbe.push_back(&be[i]);
  std::stable_sort(qrt.begin(), qrt.end(), [](auto a, auto b) { return a->remaining_us < b->remaining_us; });
  std::stable_sort(qbe.begin(), qbe.end(), [](auto a, auto b) { return a->m_cpu < b->m_cpu; });
  return schedule_ordered(as_mgr(mgr), qrt, qbe, batch_size, cost, rt_ready, n_rt_ready, be_ready, n_be_ready,
                          over_budget);
}

int bros_schedule_pulled(void* mgr, const bros_sched_req* pending, int32_t n_pending, const bros_sched_req* waiting,
                         int32_t n_waiting, const bros_sched_req* be, int32_t n_be, int32_t batch_size,
                         const bros_cost_model* cost, int32_t* rt_ready, int32_t* n_rt_ready, int32_t* be_ready,
                         int32_t* n_be_ready, int32_t* over_budget) {
  const char* fn = "bros_schedule_pulled";
  if (!mgr || !cost || !rt_ready || !n_rt_ready || !be_ready || !n_be_ready || !over_budget)
    return fail(BROS_E_NULL, "%s: NULL argument", fn);
  if ((n_pending > 0 && !pending) || (n_waiting > 0 && !waiting) || (n_be > 0 && !be) || n_pending < 0 ||
      n_waiting < 0 || n_be < 0 || batch_size < 0)
    return fail(BROS_E_SHAPE, "%s: bad queue arguments", fn);
  // Only the pending queue is sorted, and only as far as the batch can reach;
  // the waiting queue is taken in its own order. Polling the two heads and
  // pulling the more urgent one yields the RT order Alg. 1 consumes.
  const size_t k = (size_t)batch_size;
  std::vector<const bros_sched_req*> qp;
  qp.reserve(n_pending);
  for (int32_t i = 0; i < n_pending; ++i) qp.push_back(&pending[i]);
  first_k_sorted(qp, k, [](const bros_sched_req* r) { return r->remaining_us; });
  std::vector<const bros_sched_req*> qrt;
  qrt.reserve(std::min(k, qp.size() + (size_t)n_waiting));
  size_t ip = 0, iw = 0;
  while (qrt.size() < k && (ip < qp.size() || iw < (size_t)n_waiting)) {
    const bool take_pending =
        iw >= (size_t)n_waiting || (ip < qp.size() && qp[ip]->remaining_us <= waiting[iw].remaining_us);
    qrt.push_back(take_pending ? qp[ip++] : &waiting[iw++]);
  }
  std::vector<const bros_sched_req*> qbe;
  qbe.reserve(n_be);
  for (int32_t i = 0; i < n_be; ++i) qbe.push_back(&be[i]);
  first_k_sorted(qbe, 2 * k + 1, [](const bros_sched_req* r) { return r->m_cpu; });
  return schedule_ordered(as_mgr(mgr), qrt, qbe, batch_size, cost, rt_ready, n_rt_ready, be_ready, n_be_ready,
                          over_budget);
}

int32_t bros_next_batch_size(int32_t current, int32_t base, int32_t max_size, int32_t over_budget) {
  if (over_budget) return base;                         // aggressive backoff
  const int64_t grown = (int64_t)current * 2;           // gradual expansion
  return (int32_t)std::min<int64_t>(grown, max_size);
}

}  // extern "C"
