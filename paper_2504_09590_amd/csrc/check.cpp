// bros_check_batch: host-side consistency check of one batch's metadata.
//
// Two sequences may share a block (an RT tail from the left end, a BE tail
// from the right end, Sec. 5.1), but a consistent batch never maps two valid
// (sequence, position) pairs to one (block, slot): the paper checkpoints a
// peer's token before it is overwritten (Sec. 5.2). This checker is pure C++
// and runs on host copies; the kernels rely on it rather than re-validating
// tables on the device.
#include "bros_attn.h"
#include "bros_error.h"

#include <cstdint>
#include <vector>

using bros::fail;

extern "C" int bros_check_batch(const int32_t* block_tables, int32_t max_blocks_per_seq,
                                const int8_t* dir, const uint8_t* cls, int32_t dir_per_entry, const int32_t* ctx_lens,
                                int32_t num_seqs, int32_t num_blocks, int32_t block_size,
                                int32_t check_slot_disjointness) {
  if (block_size != 16) return fail(BROS_E_UNSUPPORTED, "block_size %d unsupported (16 only)", block_size);
  if (num_seqs < 0 || max_blocks_per_seq <= 0 || num_blocks <= 0)
    return fail(BROS_E_SHAPE, "bad counts: num_seqs=%d max_blocks_per_seq=%d num_blocks=%d", num_seqs, max_blocks_per_seq, num_blocks);
  if (num_seqs == 0) return bros::ok();
  if (!block_tables || !ctx_lens) return fail(BROS_E_NULL, "block_tables or ctx_lens is NULL");
  if (!dir && !cls) return fail(BROS_E_NULL, "dir and cls are both NULL");

  if (dir_per_entry != 0 && dir_per_entry != 1) return fail(BROS_E_SHAPE, "dir_per_entry %d is neither 0 nor 1", dir_per_entry);
  if (dir_per_entry && !dir) return fail(BROS_E_NULL, "dir_per_entry is set but dir is NULL");
  // Direction of table entry b of sequence s (validated below).
  auto dir_of = [&](int s, int b) -> int {
    if (!dir) return cls[s] == 1 ? -1 : 1;
    return dir_per_entry ? dir[(size_t)s * max_blocks_per_seq + b] : dir[s];
  };
  std::vector<int> d(num_seqs);
  for (int s = 0; s < num_seqs; ++s) {
    if (dir && !dir_per_entry) {
      if (dir[s] != 1 && dir[s] != -1) return fail(BROS_E_TABLE, "sequence %d: direction flag %d is not +1 or -1", s, (int)dir[s]);
      d[s] = dir[s];
    } else if (dir) {
      d[s] = 1;   // per entry: checked with the table below
    } else {
      if (cls[s] > 1) return fail(BROS_E_TABLE, "sequence %d: class %u is neither RT (0) nor BE (1)", s, (unsigned)cls[s]);
      d[s] = cls[s] == 1 ? -1 : 1;
    }
    if (ctx_lens[s] < 0) return fail(BROS_E_TABLE, "sequence %d: negative context %d", s, ctx_lens[s]);
    if ((int64_t)ctx_lens[s] > (int64_t)max_blocks_per_seq * 16)
      return fail(BROS_E_TABLE, "sequence %d: context %d exceeds %d table entries", s, ctx_lens[s], max_blocks_per_seq);
    const int nblk = (ctx_lens[s] + 15) / 16;
    for (int b = 0; b < nblk; ++b) {
      const int32_t id = block_tables[(size_t)s * max_blocks_per_seq + b];
      if (id < 0 || id >= num_blocks)
        return fail(BROS_E_TABLE, "sequence %d: table entry %d = %d outside [0, %d)", s, b, id, num_blocks);
      if (dir_per_entry) {
        const int f = dir[(size_t)s * max_blocks_per_seq + b];
        if (f != 1 && f != -1) return fail(BROS_E_TABLE, "sequence %d entry %d: direction flag %d is not +1 or -1", s, b, f);
      }
    }
  }
  if (!check_slot_disjointness) return bros::ok();

  // One bit per (block, slot); positions < ctx of every sequence must be unique.
  std::vector<uint16_t> used((size_t)num_blocks, 0);
  for (int s = 0; s < num_seqs; ++s) {
    for (int p = 0; p < ctx_lens[s]; ++p) {
      const int32_t id = block_tables[(size_t)s * max_blocks_per_seq + p / 16];
      const int off = p % 16;
      const int slot = (dir_per_entry ? dir_of(s, p / 16) : d[s]) > 0 ? off : 15 - off;
      const uint16_t bit = (uint16_t)(1u << slot);
      if (used[id] & bit)
        return fail(BROS_E_TABLE, "sequence %d position %d: block %d slot %d is already owned by another token", s, p, id, slot);
      used[id] |= bit;
    }
  }
  return bros::ok();
}

// A scatter's slot list: ids inside the pool must be distinct, else two rows
// race for one slot.
extern "C" int bros_check_slot_ids(const int32_t* slot_ids, int32_t num_slots, int32_t num_blocks) {
  if (num_slots < 0 || num_blocks <= 0)
    return fail(BROS_E_SHAPE, "bad counts: num_slots=%d num_blocks=%d", num_slots, num_blocks);
  if (num_slots == 0) return bros::ok();
  if (!slot_ids) return fail(BROS_E_NULL, "slot_ids is NULL");
  const int64_t pool_slots = (int64_t)num_blocks * 16;
  std::vector<uint8_t> seen((size_t)pool_slots, 0);
  for (int32_t i = 0; i < num_slots; ++i) {
    const int64_t id = slot_ids[i];
    if (id < 0 || id >= pool_slots) continue;
    if (seen[(size_t)id]) return fail(BROS_E_TABLE, "slot id %lld (block %lld slot %lld) appears again at index %d",
                                      (long long)id, (long long)(id / 16), (long long)(id % 16), i);
    seen[(size_t)id] = 1;
  }
  return bros::ok();
}

// Slot ids (block * 16 + slot) of chosen (sequence, logical position) pairs,
// with the mapping every kernel uses: entry p / 16 of the sequence's table and
// slot p % 16 walking from the left, 15 - p % 16 from the right (Sec. 5.1,
// with the exclusive view of Sec. 5.2).
extern "C" int bros_slot_ids(const int32_t* block_tables, int32_t max_blocks_per_seq, const int8_t* dir,
                             const uint8_t* cls, int32_t dir_per_entry, int32_t num_seqs, int32_t num_blocks,
                             const int32_t* seqs, const int32_t* positions, int32_t n, int32_t* slot_ids) {
  if (num_seqs < 0 || max_blocks_per_seq <= 0 || num_blocks <= 0 || n < 0)
    return fail(BROS_E_SHAPE, "bad counts: num_seqs=%d max_blocks_per_seq=%d num_blocks=%d n=%d", num_seqs,
                max_blocks_per_seq, num_blocks, n);
  if (n == 0) return bros::ok();
  if (!block_tables || !seqs || !positions || !slot_ids) return fail(BROS_E_NULL, "a table, list or output pointer is NULL");
  if (!dir && !cls) return fail(BROS_E_NULL, "dir and cls are both NULL");
  if (dir_per_entry != 0 && dir_per_entry != 1) return fail(BROS_E_SHAPE, "dir_per_entry %d is neither 0 nor 1", dir_per_entry);
  if (dir_per_entry && !dir) return fail(BROS_E_NULL, "dir_per_entry is set but dir is NULL");
  for (int32_t i = 0; i < n; ++i) {
    const int s = seqs[i], p = positions[i];
    if (s < 0 || s >= num_seqs) return fail(BROS_E_TABLE, "pair %d: sequence %d outside [0, %d)", i, s, num_seqs);
    if (p < 0 || p / 16 >= max_blocks_per_seq)
      return fail(BROS_E_TABLE, "pair %d: position %d beyond the %d table entries", i, p, max_blocks_per_seq);
    const int32_t id = block_tables[(size_t)s * max_blocks_per_seq + p / 16];
    if (id < 0 || id >= num_blocks)
      return fail(BROS_E_TABLE, "pair %d: sequence %d entry %d = %d outside [0, %d)", i, s, p / 16, id, num_blocks);
    int d;
    if (!dir) {
      d = cls[s] == 1 ? -1 : 1;
    } else {
      d = dir_per_entry ? dir[(size_t)s * max_blocks_per_seq + p / 16] : dir[s];
      if (d != 1 && d != -1) return fail(BROS_E_TABLE, "pair %d: direction flag %d is not +1 or -1", i, d);
    }
    const int off = p % 16;
    slot_ids[i] = id * 16 + (d > 0 ? off : 15 - off);
  }
  return bros::ok();
}
