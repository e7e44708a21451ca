// Per-XCD work queues of the large-tile grouped-GEMM kernels (tiled and big-tile classes).
//
// Workgroup b runs on XCD b % 8 (round-robin placement).  Items (token tile, feature block)
// are grouped in chunks of tg token tiles x fg feature blocks (tg * fg = the workgroups of one
// XCD), so one XCD's L2 is shared by tg token tiles and fg weight blocks instead of every token
// tile being spread over all XCDs.  The chunks form one work queue per XCD (chunk c in queue
// c % 8, in order), taken item by item through an atomic ticket: the items an XCD runs at one
// time are then always neighbours in chunk order, however far its workgroups drift apart (a
// fixed round-robin assignment let them drift whole chunks apart over the rounds, and the
// sharing with them).  A workgroup whose queue is empty takes items from the next XCDs' queues.
//
// The queue words are control words kQueueCtrl .. + kXcds (tickets, then the count of finished
// workgroups).  They are zero between launches: the routing kernel clears them and the last
// workgroup out of each launch returns them to zero.  Nothing waits on another workgroup: a
// take tries at most one ticket per queue once it is empty.
#pragma once

#include "common.h"

namespace damoe {

constexpr int kXcds = 8;

struct ItemMap {
  bool xcd;
  int fg, tg, n_fg, nq, n_chunks;

  __device__ ItemMap(int n_tiles, int n_fb) {
    const int per_xcd = gridDim.x / kXcds;
    xcd = gridDim.x % kXcds == 0 && per_xcd > 0;
    fg = n_fb % 4 == 0 ? 4 : n_fb % 2 == 0 ? 2 : 1;
    if (!xcd || fg > per_xcd) fg = 1;
    tg = xcd ? per_xcd / fg : 1;
    n_fg = n_fb / fg;
    nq = xcd ? kXcds : 1;
    n_chunks = (n_tiles + tg - 1) / tg * n_fg;
  }

  // Tickets of queue q: its chunks q, q + nq, ... times tg * fg items each.
  __device__ int queue_len(int q) const { return q < n_chunks ? ((n_chunks - 1 - q) / nq + 1) * (tg * fg) : 0; }

  // Item of ticket t of queue q; false for the slots past the last tile of a partial chunk.
  __device__ bool item(int q, int t, int n_tiles, int& tile, int& fb) const {
    const int chunk = q + t / (tg * fg) * nq;
    const int local = t % (tg * fg);
    const int tgroup = chunk / n_fg;
    tile = tgroup * tg + local / fg;
    fb = (chunk - tgroup * n_fg) * fg + local % fg;
    return tile < n_tiles;
  }
};

// Thread 0's side of the queues.  take() returns queue << 28 | ticket, or -1 once every queue
// is empty; the workgroup learns it through an LDS word (the kernels' item loops).  A
// workgroup's first ticket is fixed: ticket blockIdx.x / nq of its own queue, so that the
// first items spread over the workgroups in launch order, one per CU while there are fewer
// items than CUs (taken first-come, two could land on one CU and leave another idle); the
// counters hand out the tickets after those.
struct QueueTaker {
  uint32_t* qctrl;
  int qj = 0;          // queues found empty so far, own queue first
  bool first = true;

  __device__ explicit QueueTaker(int32_t* ctrl) : qctrl(reinterpret_cast<uint32_t*>(ctrl + kQueueCtrl)) {}

  __device__ int take(const ItemMap& m) {
    const int fixed = (int)gridDim.x / m.nq;  // tickets per queue taken as first tickets
    if (first) {
      first = false;
      const int q = (int)blockIdx.x % m.nq, t = (int)blockIdx.x / m.nq;
      if (t < m.queue_len(q)) return q << 28 | t;
    }
    while (qj < m.nq) {
      const int q = ((int)blockIdx.x + qj) % m.nq;
      const int t = fixed + (int)atomicAdd(qctrl + q, 1u);
      if (t < m.queue_len(q)) return q << 28 | t;
      ++qj;
    }
    return -1;
  }

  // After the workgroup's last take: the last workgroup out returns the words to zero (every
  // other workgroup has finished taking tickets, its last ticket returned before its count).
  __device__ void finish() {
    const uint32_t done = atomicAdd(qctrl + kXcds, 1u);
    if (done == gridDim.x - 1) {
      for (int x = 0; x <= kXcds; ++x) __hip_atomic_store(qctrl + x, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
};

}  // namespace damoe
