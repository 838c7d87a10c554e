// Multi-replica admission of the shared Waiting queue (host code, no GPU work).
//
// Each replica keeps its own GPU and CPU queues and one Waiting queue is shared
// by all of them (Sec. 4.1).  Programs promoted from a replica's CPU tier stay
// on that replica (cache affinity) and are handled by its own plan; Waiting
// programs have no KV anywhere and are bin-packed across the replicas' free
// GPU capacity (Sec. 4.3.1): candidates in decreasing size, each onto the
// replica with the most room that holds it, or with MORI_ADMIT_BEST_FIT onto
// the one with the least such room.  The free rooms live in an ordered set, so
// each choice is a logarithmic lookup.
#include <algorithm>
#include <cstring>
#include <set>
#include <utility>
#include <vector>

#include "mori.h"

extern "C" int mori_replica_admit(uint32_t num_programs, const uint64_t* bytes, const float* idleness,
                                  const uint8_t* status, uint32_t num_replicas, const uint64_t* room,
                                  uint32_t flags, int32_t* replica, uint64_t* room_after) {
  const uint32_t P = num_programs, R = num_replicas;
  if (R == 0 || R > MORI_MAX_REPLICAS || !room || !room_after) return MORI_EINVAL;
  if (P && (!bytes || !idleness || !status || !replica)) return MORI_EINVAL;
  if (flags & ~MORI_ADMIT_BEST_FIT) return MORI_EINVAL;
  for (uint32_t p = 0; p < P; ++p)
    if (status[p] > MORI_ST_NEW || !(idleness[p] >= 0.0f && idleness[p] <= 1.0f)) return MORI_EINVAL;

  std::vector<uint32_t> cand;
  cand.reserve(P);
  for (uint32_t p = 0; p < P; ++p) {
    replica[p] = -1;
    if (status[p] != MORI_ST_ACTING) cand.push_back(p);  // Acting: in a tool call, nothing to admit
  }
  // returning programs before new arrivals; larger KV first; lower idleness; lower id
  std::sort(cand.begin(), cand.end(), [&](uint32_t x, uint32_t y) {
    const bool nx = status[x] == MORI_ST_NEW, ny = status[y] == MORI_ST_NEW;
    if (nx != ny) return ny;
    if (bytes[x] != bytes[y]) return bytes[x] > bytes[y];
    if (idleness[x] != idleness[y]) return idleness[x] < idleness[y];
    return x < y;
  });

  std::memmove(room_after, room, sizeof(uint64_t) * R);
  std::set<std::pair<uint64_t, uint32_t>> free_room;  // (room, replica), ascending
  for (uint32_t r = 0; r < R; ++r) free_room.emplace(room_after[r], r);
  const bool best_fit = (flags & MORI_ADMIT_BEST_FIT) != 0;
  for (const uint32_t p : cand) {
    const uint64_t b = bytes[p];
    auto it = free_room.end();
    if (best_fit) {
      it = free_room.lower_bound({b, 0u});  // least room that holds it, lowest replica on ties
    } else {
      const uint64_t most = free_room.rbegin()->first;
      if (most >= b) it = free_room.lower_bound({most, 0u});  // most room, lowest replica on ties
    }
    if (it == free_room.end()) continue;  // fits nowhere: stays waiting
    const uint32_t r = it->second;
    free_room.erase(it);
    room_after[r] -= b;
    free_room.emplace(room_after[r], r);
    replica[p] = static_cast<int32_t>(r);
  }
  return MORI_OK;
}
