// CPU driver for the union-find walks of tg_mask_rois (csrc/unionfind.h), run by
// test_unionfind.py. Reads one case per line from stdin and prints one result line:
//   F n p_0 .. p_{n-1} i       -> "<root or -1> <parent() calls>"
//   U n p_0 .. p_{n-1} a b     -> "<1 or 0> <parent() calls> q_0 .. q_{n-1}" (array after)
//   X n p_0 .. p_{n-1} a b v   -> as U, but the first link() reports v as the link it
//                                 replaced, as if another thread had written v there
//   E n m a_0 b_0 .. a_m b_m   -> from the identity array, unite every edge in order;
//                                 "<all ok> r_0 .. r_{n-1} q_0 .. q_{n-1}" with r_i the
//                                 find of i after all edges and q the array
// The accessor counts parent() reads so that the tests can bound the work of a walk over
// a broken array.
#include <cstdio>
#include <vector>

#include "unionfind.h"

namespace {

struct Plain {
  std::vector<int> a;
  long reads = 0;
  bool planted = false;
  int plant = 0;
  int parent(int i) {
    ++reads;
    return a[i];
  }
  int link(int i, int p) {
    const int old = a[i];
    if (p < old) a[i] = p;
    if (planted) {
      planted = false;
      return plant;
    }
    return old;
  }
};

bool read_array(int n, Plain &m) {
  m.a.resize(n);
  for (int k = 0; k < n; ++k)
    if (std::scanf("%d", &m.a[k]) != 1) return false;
  return true;
}

void print_array(const Plain &m) {
  for (int v : m.a) std::printf(" %d", v);
}

}  // namespace

int main() {
  char op;
  while (std::scanf(" %c", &op) == 1) {
    int n = 0;
    if (std::scanf("%d", &n) != 1 || n < 1) return 2;
    Plain m;
    if (op == 'F') {
      int i;
      if (!read_array(n, m) || std::scanf("%d", &i) != 1) return 2;
      const int r = tg_detail::uf_find(m, i);
      std::printf("%d %ld\n", r, m.reads);
    } else if (op == 'U') {
      int a, b;
      if (!read_array(n, m) || std::scanf("%d %d", &a, &b) != 2) return 2;
      const bool ok = tg_detail::uf_unite(m, a, b);
      std::printf("%d %ld", ok ? 1 : 0, m.reads);
      print_array(m);
      std::printf("\n");
    } else if (op == 'X') {
      int a, b;
      if (!read_array(n, m) || std::scanf("%d %d %d", &a, &b, &m.plant) != 3) return 2;
      m.planted = true;
      const bool ok = tg_detail::uf_unite(m, a, b);
      std::printf("%d %ld", ok ? 1 : 0, m.reads);
      print_array(m);
      std::printf("\n");
    } else if (op == 'E') {
      int e;
      if (std::scanf("%d", &e) != 1) return 2;
      m.a.resize(n);
      for (int k = 0; k < n; ++k) m.a[k] = k;
      bool ok = true;
      for (int k = 0; k < e; ++k) {
        int a, b;
        if (std::scanf("%d %d", &a, &b) != 2) return 2;
        ok = tg_detail::uf_unite(m, a, b) && ok;
      }
      std::printf("%d", ok ? 1 : 0);
      for (int k = 0; k < n; ++k) std::printf(" %d", tg_detail::uf_find(m, k));
      print_array(m);
      std::printf("\n");
    } else {
      return 2;
    }
  }
  return 0;
}
