// Host-side declarations of the scheduler-step kernel (csrc/pa_sched.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

// Scheduler step (page allocator and block-table builder): one workgroup of
// kSchedThreads threads, each holding up to 8 slots.
constexpr int kSchedThreads = 1024;
constexpr int kSchedMaxSlots = 8 * kSchedThreads;

struct SchedArgs {
  int32_t* free_pages;
  int32_t* hdr;
  int32_t* queue_seq;
  int32_t* queue_tok;
  int32_t* queue_fin;
  int32_t* slot_seq;
  int32_t* slot_order;
  int32_t* slot_fin;
  int32_t* context_lens;
  int32_t* block_table;
  int S, P, MP, Q, n_real;
  const int32_t* new_seq;
  const int32_t* new_prompt;
  const int32_t* new_fin;
  int n_new;
  int32_t* query_start_loc;
  int32_t* finished_out;
  int32_t* info;
};

int sched_slots_per_thread(int S);  // 1, 2, 4, 8, or 0 if S > kSchedMaxSlots
hipError_t launch_sched(const SchedArgs& a, hipStream_t st);

}  // namespace pa
