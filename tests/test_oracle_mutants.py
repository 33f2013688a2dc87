"""The oracle's pins catch plausible mistakes (no GPU).

Each case below plants one mistake in a copy of oracle/oracle.c (a dropped
term, a wrong comparison, a swapped axis, a wrong constant), builds it with
gcc in a temporary directory, and runs the oracle pin tests against that
build in a child process.  The pins must fail for every mutant.
"""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
DBSCAN_PINS = "tests/test_oracle_dbscan.py"
KDE_PINS = "tests/test_oracle_kde.py"
HEAT_PINS = "tests/test_oracle_heatmap.py"
ROI_PINS = "tests/test_oracle_roi.py"
DRINK_PINS = "tests/test_oracle_drinkers.py"
MASK_PINS = "tests/test_oracle_mask.py"

MUTANTS = [
    # (name, old text, new text, which pin file must fail)
    ("strict_ball", "if (sq_dist(xy, i, j) <= e2) ++c;\n        count[i] = c;\n        core[i]",
     "if (sq_dist(xy, i, j) < e2) ++c;\n        count[i] = c;\n        core[i]", DBSCAN_PINS),
    ("self_not_counted", "if (sq_dist(xy, i, j) <= e2) ++c;\n        count[i] = c;\n        core[i]",
     "if (j != i && sq_dist(xy, i, j) <= e2) ++c;\n        count[i] = c;\n        core[i]",
     DBSCAN_PINS),
    ("core_strict", "c >= (int64_t)min_pts", "c > (int64_t)min_pts", DBSCAN_PINS),
    ("expand_through_border", "if (core[j] && comp[j] < 0 && sq_dist(xy, p, j) <= e2)",
     "if (comp[j] < 0 && sq_dist(xy, p, j) <= e2)", DBSCAN_PINS),
    ("seeds_descending", "for (int32_t s = 0; s < n; ++s) {",
     "for (int32_t s = n - 1; s >= 0; --s) {", DBSCAN_PINS),
    ("border_first_core", "else if (d2 != best_d2) better = d2 < best_d2;", "", DBSCAN_PINS),
    ("border_x_before_y",
     "else if (xy[2 * j + 1] != xy[2 * best + 1]) better = xy[2 * j + 1] < xy[2 * best + 1];\n"
     "            else better = xy[2 * j] < xy[2 * best];",
     "else if (xy[2 * j] != xy[2 * best]) better = xy[2 * j] < xy[2 * best];\n"
     "            else better = xy[2 * j + 1] < xy[2 * best + 1];", DBSCAN_PINS),
    ("border_larger_y", "better = xy[2 * j + 1] < xy[2 * best + 1];",
     "better = xy[2 * j + 1] > xy[2 * best + 1];", DBSCAN_PINS),
    ("dy_uses_x", "int64_t dy = (int64_t)xy[2 * i + 1] - (int64_t)xy[2 * j + 1];",
     "int64_t dy = (int64_t)xy[2 * i] - (int64_t)xy[2 * j + 1];", DBSCAN_PINS),
    ("kde_no_half_cell", "const double cx = ((double)gx + 0.5)", "const double cx = ((double)gx)",
     KDE_PINS),
    ("kde_norm_2pi_sigma", "return acc / (kPi * two_s2);", "return acc / (kPi * sigma_px * 2.0);",
     KDE_PINS),
    ("kde_sigma_sq_not_doubled", "const double two_s2 = 2.0 * sigma_px * sigma_px;",
     "const double two_s2 = sigma_px * sigma_px;", KDE_PINS),
    ("kde_quantum_8", "const double x = (double)xy[2 * i] / 16.0;",
     "const double x = (double)xy[2 * i] / 8.0;", KDE_PINS),
    ("kde_axes_swapped", "const double dx = cx - x, dy = cy - y;",
     "const double dx = cx - y, dy = cy - x;", KDE_PINS),
    ("kde_cy_uses_width", "const double cy = ((double)gy + 0.5) * (double)height_px",
     "const double cy = ((double)gy + 0.5) * (double)width_px", KDE_PINS),
    ("kde_row_layout", "double *row = job->density + ((int64_t)f * job->grid_h + gy) * job->grid_w;",
     "double *row = job->density + ((int64_t)f * job->grid_w + gy) * job->grid_h;", KDE_PINS),
    ("heat_strict_threshold", "if (!(density[seed] >= threshold) || labels[seed] >= 0) continue;",
     "if (!(density[seed] > threshold) || labels[seed] >= 0) continue;", HEAT_PINS),
    ("heat_4_as_8", "if (connectivity == 4 && dx != 0 && dy != 0) continue;", "", HEAT_PINS),
    ("heat_seeds_descending", "for (int64_t seed = 0; seed < cells; ++seed) {",
     "for (int64_t seed = cells - 1; seed >= 0; --seed) {", HEAT_PINS),
    ("heat_entropy_log2", "H -= pc * log(pc);", "H -= pc * log2(pc);", HEAT_PINS),
    ("heat_entropy_unnormalised", "const double pc = (double)density[c] / S;",
     "const double pc = (double)density[c];", HEAT_PINS),
    ("heat_degree_counts", "if (labels[c] >= 0) hot += (double)density[c];",
     "if (labels[c] >= 0) hot += 1.0;", HEAT_PINS),
    ("heat_degree_not_normalised", "*degree = S > 0.0 ? hot / S : 0.0;", "*degree = S > 0.0 ? hot : 0.0;",
     HEAT_PINS),
    ("heat_mass_no_area", "for (int64_t c = 0; c < cells; ++c) comp_mass[c] *= cell_area;", "", HEAT_PINS),
    ("heat_mass_at_cell", "comp_mass[labels[c]] += (double)density[c];", "comp_mass[c] += (double)density[c];",
     HEAT_PINS),
    ("roi_open_boundary", "if (on_segment(px, py, ax, ay, bx, by)) return 1;", "", ROI_PINS),
    ("roi_segment_unbounded", "return px >= lo_x && px <= hi_x && py >= lo_y && py <= hi_y;", "return 1;",
     ROI_PINS),
    ("roi_vertex_on_ray_twice", "if ((ay > py) != (by > py)) {", "if ((ay >= py) != (by > py)) {", ROI_PINS),
    ("roi_no_flip", "const int right = (by > ay) ? (lhs < rhs) : (lhs > rhs);", "const int right = lhs < rhs;",
     ROI_PINS),
    ("roi_axes_swapped", "if (!oracle_point_in_polygon(poly, n_vertices, xy[2 * i], xy[2 * i + 1])) continue;",
     "if (!oracle_point_in_polygon(poly, n_vertices, xy[2 * i + 1], xy[2 * i])) continue;", ROI_PINS),
    ("roi_counts_cumulative", "counts[f] = c;\n        out_offsets[f + 1] = k;",
     "counts[f] = k;\n        out_offsets[f + 1] = k;", ROI_PINS),
    ("drink_at_threshold", "if (len2 == 0 || dot <= 0) return wx * wx + wy * wy < t2;",
     "if (len2 == 0 || dot <= 0) return wx * wx + wy * wy <= t2;", DRINK_PINS),
    ("drink_no_clamp_a", "if (len2 == 0 || dot <= 0) return wx * wx + wy * wy < t2;",
     "if (len2 == 0) return wx * wx + wy * wy < t2;", DRINK_PINS),
    ("drink_no_clamp_b", "if (dot >= len2) {", "if (0) {", DRINK_PINS),
    ("drink_threshold_not_squared", "const unsigned __int128 lim = (unsigned __int128)t2 * (unsigned __int128)len2;",
     "const unsigned __int128 lim = (unsigned __int128)t * (unsigned __int128)len2;", DRINK_PINS),
    ("drink_last_index", "for (int32_t k = 0; k < n_lines && hit < 0; ++k)", "for (int32_t k = 0; k < n_lines; ++k)",
     DRINK_PINS),
    ("drink_dy_from_x", "const int64_t wx = (int64_t)px - ax, wy = (int64_t)py - ay;",
     "const int64_t wx = (int64_t)px - ax, wy = (int64_t)py - ax;", DRINK_PINS),
    ("mask_threshold_inclusive", "if (!(P[seed] > threshold) || L[seed] >= 0) continue;",
     "if (!(P[seed] >= threshold) || L[seed] >= 0) continue;", MASK_PINS),
    ("mask_4_as_8", "if (connectivity == 4 && dx * dy != 0) continue;", "", MASK_PINS),
    ("mask_seeds_descending", "for (int64_t seed = 0; seed < px; ++seed) {",
     "for (int64_t seed = px - 1; seed >= 0; --seed) {", MASK_PINS),
    ("mask_box_width_exclusive", "comp_box[4 * k + 2] = x1 - x0 + 1;", "comp_box[4 * k + 2] = x1 - x0;", MASK_PINS),
    ("mask_box_height_from_x", "comp_box[4 * k + 3] = y1 - y0 + 1;", "comp_box[4 * k + 3] = x1 - x0 + 1;",
     MASK_PINS),
    ("mask_centroid_y_from_x", "comp_centroid[2 * k + 1] = (double)sy / (double)area;",
     "comp_centroid[2 * k + 1] = (double)sx / (double)area;", MASK_PINS),
    ("mask_xy_rounded", "comp_xy[2 * k + 1] = (int32_t)((16 * sy) / area);",
     "comp_xy[2 * k + 1] = (int32_t)((16 * sy + area / 2) / area);", MASK_PINS),
    ("mask_score_of_seed", "if (P[c] > best) best = P[c];", "", MASK_PINS),
    ("mask_offsets_per_frame", "comp_offsets[f + 1] = k;", "comp_offsets[f + 1] = nc;", MASK_PINS),
]


@pytest.mark.parametrize("name,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new, pins):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mutant_c = tmp_path / "oracle_mutant.c"
    mutant_c.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-w",
                           "-o", str(lib), str(mutant_c), "-lm"])
    env = dict(os.environ, ORACLE_LIB_OVERRIDE=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", pins],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch mutant {name}:\n{r.stdout[-2000:]}"
