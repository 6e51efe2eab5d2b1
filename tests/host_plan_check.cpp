// CPU test driver for the host planning code (csrc/plan.cpp), built with the
// address and undefined-behaviour sanitizers by tests/test_host_sanitized.py.
// Reads one case per line on stdin and prints the result on one line:
//   T n prefix max_tree max_depth vocab cap tok[n] par[n]
//       -> rc depth[n] pos[n] anc[n]            (griffin tree preparation)
//   S batch splits sp prefix[batch] nodes[batch]
//       -> tab[batch*splits*4] nsplit[batch]    (prefix-attention split table)
//   D n_layers d_model hq hkv dh d_ff vocab experts top_k eps base mb mt md cap
//       -> rc                                   (model-shape validation)
//   Q batch max_tree nodes[batch] par[batch*max_tree] tok[batch*max_tree]
//       -> order | rows_with | step_child | step_token
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "plan.h"

using namespace griffin_plan;

template <typename T>
static std::vector<T> take(std::istringstream& in, long n) {
  std::vector<T> v(n > 0 ? n : 0);
  for (auto& x : v) in >> x;
  return v;
}

template <typename T>
static void put(const std::vector<T>& v) {
  for (const auto& x : v) std::cout << ' ' << x;
}

int main() {
  std::string line;
  while (std::getline(std::cin, line)) {
    std::istringstream in(line);
    char op = 0;
    in >> op;
    if (op == 'T') {
      int n, prefix, mt, md, vocab, cap;
      in >> n >> prefix >> mt >> md >> vocab >> cap;
      auto tok = take<int32_t>(in, n), par = take<int32_t>(in, n);
      tok.resize(n > 0 ? n : 1);  // non-null inputs even for an empty tree
      par.resize(n > 0 ? n : 1);
      // outputs sized exactly n: any write past them is a sanitizer error
      std::vector<int32_t> dep(n > 0 ? n : 0), pos(n > 0 ? n : 0);
      std::vector<unsigned long long> anc(n > 0 ? n : 0);
      std::string why;
      const int rc = prepare_tree(n, tok.data(), par.data(), prefix, mt, md, vocab, cap,
                                  n > 0 ? dep.data() : nullptr, n > 0 ? pos.data() : nullptr,
                                  n > 0 ? reinterpret_cast<uint64_t*>(anc.data()) : nullptr, &why);
      std::cout << rc;
      if (rc == GRIFFIN_OK) {
        put(dep);
        put(pos);
        put(anc);
      }
      std::cout << '\n';
    } else if (op == 'S') {
      int batch, splits, sp;
      in >> batch >> splits >> sp;
      auto prefix = take<int32_t>(in, batch), nodes = take<int32_t>(in, batch);
      std::vector<int32_t> tab((size_t)batch * splits * 4, 7777), nsplit(batch, 7777);
      attn_split_plan(batch, prefix.data(), nodes.data(), splits, sp, tab.data(), nsplit.data());
      put(tab);
      put(nsplit);
      std::cout << ' ' << merge_slots(nsplit.data(), batch, sp) << '\n';
    } else if (op == 'D') {
      griffin_model_desc d{};
      in >> d.n_layers >> d.d_model >> d.n_q_heads >> d.n_kv_heads >> d.head_dim >> d.d_ff >> d.vocab >>
          d.n_experts >> d.top_k >> d.rms_eps >> d.rope_base >> d.max_batch >> d.max_tree >> d.max_depth >>
          d.kv_capacity;
      std::string why;
      std::cout << validate_desc(&d, &why) << '\n';
    } else if (op == 'Q') {
      int batch, mt;
      in >> batch >> mt;
      auto nodes = take<int32_t>(in, batch);
      auto par = take<int32_t>(in, (long)batch * mt), tok = take<int32_t>(in, (long)batch * mt);
      std::vector<int32_t> order, child, token;
      std::vector<int> rows_with;
      sampled_plan(batch, mt, nodes.data(), par.data(), tok.data(), order, rows_with, child, token);
      put(order);
      std::cout << " |";
      put(rows_with);
      std::cout << " |";
      put(child);
      std::cout << " |";
      put(token);
      std::cout << '\n';
    }
  }
  return 0;
}
