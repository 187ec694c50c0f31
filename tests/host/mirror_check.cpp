// Host harness for the library's host code (built with g++ under the
// address, undefined-behaviour and thread sanitizers; see
// tests/test_host_sanitized.py).  It compiles the pool's host source itself
// against a host-only HIP stand-in (tests/host/hip/hip_runtime.h), with
// launch functions that do nothing: what runs is exactly the library's
// validation, host mirror (allocation rule, forks, frees), planner (with its
// host threads) and staging copies into the caller's workspace.
//
// Protocol: one operation per input line, one JSON object per output line.
//   create NB HQ HKV T MAXB SPLITS      a bf16 pool (workspace, tables in host memory)
//   alloc  t n [t n ...]                gambit_kv_alloc
//   write  t pos0 n                     gambit_kv_write (dummy K/V pointers)
//   fork   p c [p c ...]                gambit_kv_fork
//   free   t [t ...]                    gambit_kv_free
//   decode t [t ...]                    gambit_decode_attn, then the plan it launched
//   state                               lengths, rows, refcounts and free count of the mirror
// Every reply carries the call's status; a failed call must change nothing
// (the Python side checks the following state against its model).
#include "../../paper_2608_08020_amd/csrc/gambit_pool.cpp"

#include <iostream>
#include <sstream>

namespace gambit {
hipError_t launch_pool_init(const DevPool&, hipStream_t) { return hipSuccess; }
hipError_t launch_alloc(const DevPool&, const int32_t*, const int32_t*, int32_t, int32_t, float, bool, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_write(const DevPool&, int32_t, int32_t, int32_t, const void*, const void*, const float*,
                        hipStream_t) {
  return hipSuccess;
}
hipError_t launch_free(const DevPool&, const int32_t*, int32_t, int32_t, hipStream_t) { return hipSuccess; }
hipError_t launch_fork(const DevPool&, const int32_t*, int32_t, int32_t*, int32_t*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_attention_units(const DevPool&, const AttnLaunch&, hipStream_t) { return hipSuccess; }
hipError_t launch_attention_merge(const DevPool&, const AttnLaunch&, hipStream_t) { return hipSuccess; }
hipError_t launch_probe_rank(const ProbeLaunch&, hipStream_t) { return hipSuccess; }
hipError_t launch_rank_topk(int32_t, const int32_t*, const float*, int32_t, int32_t*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_score_update(const DevPool&, const ScoreLaunch&, hipStream_t) { return hipSuccess; }
hipError_t launch_evict_pick(const DevPool&, const int32_t*, int32_t, int32_t*, hipStream_t) { return hipSuccess; }
hipError_t launch_tournament(const DevPool&, int32_t, int32_t, int32_t, int32_t*, int32_t*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_mlp_score(const MlpLaunch&, hipStream_t) { return hipSuccess; }
hipError_t launch_record_scores(const DevPool&, const int32_t*, const float*, int32_t, hipStream_t) {
  return hipSuccess;
}
}  // namespace gambit

namespace {

struct Buffers {
  std::vector<uint8_t> kc, vc, ws_raw;
  std::vector<int32_t> table, seq, ref;
};

void print_ints(std::ostream& o, const int32_t* a, size_t n) {
  o << "[";
  for (size_t i = 0; i < n; ++i) o << (i ? "," : "") << a[i];
  o << "]";
}

void dump_state(gambit_pool* p) {
  std::ostringstream o;
  o << "{\"op\":\"state\",\"nfree\":" << p->nfree << ",\"seq_len\":";
  print_ints(o, p->seq_len.data(), p->seq_len.size());
  o << ",\"refcount\":";
  print_ints(o, p->refcount.data(), p->refcount.size());
  o << ",\"rows\":[";
  for (size_t t = 0; t < p->table.size(); ++t) {
    o << (t ? "," : "");
    print_ints(o, p->table[t].data(), p->table[t].size());
  }
  o << "]}";
  std::cout << o.str() << "\n";
}

// The plan the last decode step launched, read back from the workspace it
// was staged into, with the mirror's rows as the kernel would have read them.
void dump_plan(gambit_pool* p, int st) {
  std::ostringstream o;
  o << "{\"op\":\"decode\",\"status\":" << st;
  if (st == GAMBIT_OK) {
    const int n = (int)p->plan_list.size();
    const AttnUnit* U = ws_ptr<AttnUnit>(p, p->L.units);
    const int32_t* mem = ws_ptr<int32_t>(p, p->L.members);
    const int32_t* nk = ws_ptr<int32_t>(p, p->L.nk);
    const int32_t* list = ws_ptr<int32_t>(p, p->L.list);
    o << ",\"grid\":" << p->grid << ",\"kmax\":" << p->L.kmax << ",\"xcd_off\":";
    print_ints(o, p->xcd_off, 9);
    o << ",\"list\":";
    print_ints(o, list, n);
    o << ",\"nk\":";
    print_ints(o, nk, n);
    o << ",\"kinds\":";
    print_ints(o, p->plan_kinds.data(), p->plan_kinds.size());
    o << ",\"units\":[";
    for (int u = 0; u < p->n_units; ++u) {
      const AttnUnit& a = U[u];
      o << (u ? "," : "") << "[" << a.owner << "," << a.jb0 << "," << a.nblk << "," << a.kvh << "," << a.mem_off
        << "," << a.mem_cnt << "," << a.kidx << "," << a.flags << "]";
    }
    int max_mem = 0;
    for (int u = 0; u < p->n_units; ++u) max_mem = std::max(max_mem, U[u].mem_off + U[u].mem_cnt);
    o << "],\"members\":";
    print_ints(o, mem, max_mem);
    o << ",\"stats\":[" << p->stats.total_tokens << "," << p->stats.unique_tokens << "," << p->stats.unique_blocks
      << "," << p->stats.table_entries << "]";
  }
  o << "}";
  std::cout << o.str() << "\n";
}

}  // namespace

int main() {
  std::ios::sync_with_stdio(false);
  gambit_pool* p = nullptr;
  Buffers B;
  std::vector<uint16_t> dummy(1 << 16);  // K/V/q/out stand-ins: host code never reads them
  std::string line;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    std::string op;
    if (!(in >> op)) continue;
    std::vector<int32_t> a;
    for (int32_t x; in >> x;) a.push_back(x);
    int st = GAMBIT_OK;
    if (op == "create") {
      gambit_pool_desc d{};
      d.num_blocks = a[0];
      d.block_size = 16;
      d.num_q_heads = a[1];
      d.num_kv_heads = a[2];
      d.head_dim = 128;
      d.kv_dtype = GAMBIT_KV_BF16;
      d.max_traces = a[3];
      d.max_blocks_per_trace = a[4];
      d.max_splits = a[5];
      d.num_layers = 1;
      B.kc.assign(64, 0);
      B.vc.assign(64, 0);
      B.table.assign((size_t)a[3] * a[4], 0);
      B.seq.assign(a[3], 0);
      B.ref.assign(a[0], 0);
      d.k_cache = B.kc.data();
      d.v_cache = B.vc.data();
      d.block_table = B.table.data();
      d.seq_len = B.seq.data();
      d.refcount = B.ref.data();
      const size_t ws = gambit_workspace_size(&d);
      B.ws_raw.assign(ws + 256, 0);
      uintptr_t base = reinterpret_cast<uintptr_t>(B.ws_raw.data());
      d.workspace = reinterpret_cast<void*>((base + 255) / 256 * 256);
      d.workspace_bytes = ws;
      st = gambit_pool_create(&d, nullptr, &p);
      std::cout << "{\"op\":\"create\",\"status\":" << st << ",\"workspace\":" << ws << "}\n";
      continue;
    }
    if (!p) return 2;
    if (op == "alloc") {
      std::vector<int32_t> ids, nt;
      for (size_t i = 0; i + 1 < a.size(); i += 2) {
        ids.push_back(a[i]);
        nt.push_back(a[i + 1]);
      }
      st = gambit_kv_alloc(p, (int)ids.size(), ids.data(), nt.data(), nullptr);
    } else if (op == "write") {
      st = gambit_kv_write(p, a[0], a[1], a[2], dummy.data(), dummy.data(), nullptr, nullptr);
    } else if (op == "fork") {
      std::vector<int32_t> par, ch;
      for (size_t i = 0; i + 1 < a.size(); i += 2) {
        par.push_back(a[i]);
        ch.push_back(a[i + 1]);
      }
      st = gambit_kv_fork(p, (int)par.size(), par.data(), ch.data(), nullptr);
    } else if (op == "free") {
      st = gambit_kv_free(p, (int)a.size(), a.data(), nullptr);
    } else if (op == "decode") {
      st = gambit_decode_attn(p, (int)a.size(), a.data(), dummy.data(), dummy.data(), dummy.data(), dummy.data(),
                              GAMBIT_OUT_F32, 0.0883883f, nullptr);
      dump_plan(p, st);
      continue;
    } else if (op == "state") {
      dump_state(p);
      continue;
    } else {
      return 3;
    }
    std::cout << "{\"op\":\"" << op << "\",\"status\":" << st << "}\n";
  }
  if (p) gambit_pool_destroy(p);
  return 0;
}
