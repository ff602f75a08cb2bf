// Token order along a generalized Hilbert ("Gilbert") curve of a width x
// height grid, the query reordering of Sec. 4 (Fig. per-tile adaptivity):
// consecutive tokens of the order are neighbouring grid cells, so any run of
// block_q consecutive tokens covers a compact 2-D region whatever block_q is.
//
// Construction (the recursive rectangle subdivision of Cerveny's generalized
// Hilbert curve, written here as an explicit work stack): a region is a
// rectangle given by a start corner and two axis vectors, the major one (the
// direction the curve leaves through) and the minor one. The curve of a
// region starts in its start corner and ends in the corner reached by moving
// along the major axis only. A region one cell thick is walked straight. A
// region much longer than wide is cut across its major axis into two halves
// walked one after the other. Otherwise it is cut into three: the first half
// of the minor extent walked with the axes swapped (up and out), the rest of
// the minor extent over the full major length (across), and the remaining
// block walked back with both axes reversed (down). Cut points are moved by one
// cell where an odd half would leave no way to connect the parts, which is
// where the single diagonal step of some odd-sized grids comes from. Host code
// only: the result is a small table the caller copies to the device once.
#include <stdint.h>

#include <vector>

namespace avq {

namespace {

struct Region {
  int x, y;    // start corner
  int ax, ay;  // major axis vector (one of them is 0)
  int bx, by;  // minor axis vector (one of them is 0)
};

inline int sgn(int v) { return (v > 0) - (v < 0); }
inline int iabs(int v) { return v < 0 ? -v : v; }

}  // namespace

// Writes order[k] = y * width + x of the k-th cell of the curve. Returns the
// number of cells written (width * height).
long long gilbert_order(int width, int height, int32_t* order) {
  std::vector<Region> stack;
  stack.reserve(128);
  if (width >= height)
    stack.push_back({0, 0, width, 0, 0, height});
  else
    stack.push_back({0, 0, 0, height, width, 0});
  long long k = 0;
  auto emit = [&](int x, int y) { order[k++] = (int32_t)y * width + x; };
  while (!stack.empty()) {
    const Region r = stack.back();
    stack.pop_back();
    const int w = iabs(r.ax + r.ay), h = iabs(r.bx + r.by);
    const int dax = sgn(r.ax), day = sgn(r.ay);  // unit step along the major axis
    const int dbx = sgn(r.bx), dby = sgn(r.by);  // unit step along the minor axis
    if (h == 1) {
      for (int i = 0, x = r.x, y = r.y; i < w; ++i, x += dax, y += day) emit(x, y);
      continue;
    }
    if (w == 1) {
      for (int i = 0, x = r.x, y = r.y; i < h; ++i, x += dbx, y += dby) emit(x, y);
      continue;
    }
    // halves of both axes (rounded toward zero)
    int hax = r.ax / 2, hay = r.ay / 2, hbx = r.bx / 2, hby = r.by / 2;
    const int hw = iabs(hax + hay), hh = iabs(hbx + hby);
    // the parts are pushed in reverse so that they pop in walking order
    if (2 * w > 3 * h) {
      // long region: two halves along the major axis; an even first half
      // keeps the end of the first part next to the start of the second
      if ((hw & 1) && w > 2) {
        hax += dax;
        hay += day;
      }
      stack.push_back({r.x + hax, r.y + hay, r.ax - hax, r.ay - hay, r.bx, r.by});
      stack.push_back({r.x, r.y, hax, hay, r.bx, r.by});
      continue;
    }
    // up, across, down; an even minor half for the same reason
    if ((hh & 1) && h > 2) {
      hbx += dbx;
      hby += dby;
    }
    const Region up = {r.x, r.y, hbx, hby, hax, hay};
    const Region across = {r.x + hbx, r.y + hby, r.ax, r.ay, r.bx - hbx, r.by - hby};
    const Region down = {r.x + (r.ax - dax) + (hbx - dbx), r.y + (r.ay - day) + (hby - dby),
                         -hbx, -hby, -(r.ax - hax), -(r.ay - hay)};
    stack.push_back(down);
    stack.push_back(across);
    stack.push_back(up);
  }
  return k;
}

}  // namespace avq
