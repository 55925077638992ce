// Union-find walks with atomic-min linking, used by tg_mask_rois's connected-component
// labelling (the GPU union-find method of Playne and Hawick, 2018, with path halving).
//
// Invariant: a link never points to a larger index -- a root points to itself, and links
// only ever decrease (every write is an atomic min with a smaller index of the same set).
// Each step of a find therefore moves to a strictly smaller index, and each retry of a
// unite lowers the larger of its two roots, so both walks end; concurrent walks may see a
// link lowered under them but never raised. The walks also check the invariant as they
// go: a link that points upwards, or below zero, can only come from an inconsistent array
// (which the labelling never produces), and ends the walk with a failure instead of a
// loop.
//
// The walks are templates over an accessor M with
//   int parent(int i)        the link of i,
//   int link(int i, int p)   lowers the link of i to min(link, p) atomically and returns
//                            the link it replaced,
// so that the same code runs on LDS and global labels in the kernels and on a plain
// array in the CPU tests of these walks.
#ifndef TG_UNIONFIND_H
#define TG_UNIONFIND_H

#if defined(__HIPCC__)
#define TG_UF_FN __host__ __device__ inline
#else
#define TG_UF_FN inline
#endif

namespace tg_detail {

// Root of i's set, halving the path on the way (i relinked to its grandparent); -1 when
// the array breaks the invariant.
template <class M>
TG_UF_FN int uf_find(M &m, int i) {
  for (;;) {
    const int p = m.parent(i);
    if (p == i) return i;
    if (p < 0 || p > i) return -1;
    const int g = m.parent(p);
    if (g == p) return p;
    if (g < 0 || g > p) return -1;
    m.link(i, g);
    i = g;
  }
}

// Joins the sets of a and b: the larger root is linked under the smaller; if that root
// was relinked meanwhile, retry from what it now points to. False when the array breaks
// the invariant.
template <class M>
TG_UF_FN bool uf_unite(M &m, int a, int b) {
  for (;;) {
    a = uf_find(m, a);
    b = uf_find(m, b);
    if (a < 0 || b < 0) return false;
    if (a == b) return true;
    if (a > b) {
      const int t = a;
      a = b;
      b = t;
    }
    const int old = m.link(b, a);
    if (old == b) return true;
    if (old < 0 || old > b) return false;
    b = old;
  }
}

}  // namespace tg_detail

#endif  // TG_UNIONFIND_H
