// Host driver for the CPU sanitizer build of the planner (plan.cpp): scale lists, rectangles,
// Bottom-Left Fill stitching and conv5 windows (Sec. 3.1) over a grid of image sizes and pyramid
// recipes, batches and invalid arguments, with AddressSanitizer and UndefinedBehaviorSanitizer on.
// Checks the invariants every plan must satisfy; returns non-zero on a violation.
#include <cstdio>
#include <string>
#include <vector>

#include "common.h"

namespace dn {
int fail(int status, const std::string&) { return status; }  // the library's message store is not linked
}  // namespace dn

static int errors = 0;
#define CHECK(c)                                                              \
  do {                                                                        \
    if (!(c)) {                                                               \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__);    \
      ++errors;                                                               \
    }                                                                         \
  } while (0)

static void check_geom(const std::vector<dn_scale_geom>& g, const std::vector<dn::PlaneSize>* planes,
                       int ph, int pw, bool stitched) {
  for (size_t i = 0; i < g.size(); ++i) {
    const dn_scale_geom& a = g[i];
    CHECK(a.h >= 1 && a.w >= 1);
    CHECK(a.y >= 0 && a.x >= 0);
    if (planes) {
      CHECK(a.plane >= 0 && a.plane < (int)planes->size());
      if (a.plane >= 0 && a.plane < (int)planes->size()) {
        CHECK(a.y + a.rh <= (*planes)[a.plane].h && a.x + a.rw <= (*planes)[a.plane].w);
      }
    } else {
      CHECK(a.y + a.rh <= ph && a.x + a.rw <= pw);
    }
    if (stitched) CHECK((a.y | a.x | a.rh | a.rw) % 16 == 0);
    for (size_t j = 0; j < i; ++j) {  // rectangles of one plane do not overlap
      const dn_scale_geom& b = g[j];
      if (a.plane != b.plane || a.image != b.image) continue;
      const bool apart = a.y + a.rh <= b.y || b.y + b.rh <= a.y || a.x + a.rw <= b.x || b.x + b.rw <= a.x;
      if (stitched || !planes) CHECK(apart);
    }
  }
}

int main() {
  const int sides[] = {1, 2, 3, 15, 16, 17, 99, 227, 480, 640, 768, 1024, 2999, 4000};
  const double bases[] = {0.3, 1.0, 2.0};
  const int plane_sides[] = {0, 256, 1200, 2000};
  int plans = 0, rejected = 0;
  for (int H : sides)
    for (int W : sides)
      for (double base : bases)
        for (int ps : plane_sides)
          for (int aspects = 0; aspects < 2; ++aspects) {
            dn_pyramid_params p{};
            p.n_scales = 1 + (H * 7 + W) % 30;
            p.steps_per_octave = 1 + (H + W) % 10;
            p.base_scale = base;
            p.pad = (H + W) % 3 == 0 ? 0 : 16;
            p.pad_mode = (H + W) % 2;
            p.plane_h = p.plane_w = ps;
            if (aspects) {
              p.n_aspects = 2;
              p.aspects[0] = 0.5;
              p.aspects[1] = 2.0;
            }
            dn::Plan plan;
            const int st = dn::make_plan(H, W, p, plan);
            if (st != DN_OK) {
              ++rejected;
              continue;
            }
            ++plans;
            check_geom(plan.scales, &plan.planes, 0, 0, ps > 0);
            if (ps > 0 && H <= 1024 && W <= 1024 && !aspects) {
              for (int n_img : {1, 3, 16}) {
                std::vector<dn_scale_geom> items;
                int np = 0;
                if (dn::make_plan_batch(n_img, H, W, p, items, np) == DN_OK) {
                  CHECK(np >= 1 && (int)items.size() == n_img * (int)plan.scales.size());
                  check_geom(items, nullptr, ps, ps, true);
                }
              }
            }
          }
  // invalid recipes and sizes are rejected, never read out of bounds
  for (int bad = 0; bad < 8; ++bad) {
    dn_pyramid_params p{};
    p.n_scales = bad == 0 ? 0 : (bad == 1 ? 100000 : 10);
    p.steps_per_octave = bad == 2 ? 0 : 3;
    p.base_scale = bad == 3 ? -1.0 : 1.0;
    p.pad = bad == 4 ? -5 : 16;
    p.pad_mode = bad == 5 ? 9 : 1;
    p.plane_h = p.plane_w = bad == 6 ? 8 : 600;
    p.n_aspects = bad == 7 ? 100 : 0;
    dn::Plan plan;
    CHECK(dn::make_plan(768, 1024, p, plan) != DN_OK);
  }
  {
    dn_pyramid_params p{};
    p.n_scales = 3;
    p.steps_per_octave = 2;
    p.base_scale = 1.0;
    dn::Plan plan;
    CHECK(dn::make_plan(0, 10, p, plan) != DN_OK);
    CHECK(dn::make_plan(-3, 10, p, plan) != DN_OK);
    CHECK(dn::make_plan(40000, 10, p, plan) != DN_OK);
  }
  int64_t s[8];
  for (int64_t n = 0; n < 5000; ++n) {
    dn::stack_sides(n, s);
    for (int k = 0; k < 8; ++k) CHECK(s[k] >= 0 && s[k] <= n);
  }
  std::printf("plans %d, rejected %d, errors %d\n", plans, rejected, errors);
  return errors ? 1 : 0;
}
