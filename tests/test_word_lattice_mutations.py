"""The word-lattice pins must catch plausible mistakes in
oracle/word_lattice.py: each case loads a copy of the module with one
mistake planted and runs the pins against it; some pin must fail."""
import importlib.util
import os

import pytest

import test_word_lattice_oracle as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "word_lattice.py")

MUTATIONS = {
    "loglike_frame_shifted": ("stack.append((j + 1, int(g.dst[a]), f32(f32(c + w) - ll[kept[j], il - 1]), nw))",
                              "stack.append((j + 1, int(g.dst[a]), f32(f32(c + w) - ll[kept[j - 1], il - 1]), nw))"),
    "one_rounding": ("stack.append((j + 1, int(g.dst[a]), f32(f32(c + w) - ll[kept[j], il - 1]), nw))",
                     "stack.append((j + 1, int(g.dst[a]), f32(float(c) + float(w) - float(ll[kept[j], il - 1])), nw))"),
    "eps_weight_dropped": ("stack.append((j, int(g.dst[a]), f32(c + w), nw))",
                           "stack.append((j, int(g.dst[a]), f32(c), nw))"),
    "epsilon_words_dropped": ("nw = words + ((ol,) if ol != 0 else ())",
                              "nw = words + ((ol,) if ol != 0 and il != 0 else ())"),
    "final_weight_ignored": ("tot = [f32(e[1]) + f32(fw[e[0]]) for e in ends]",
                             "tot = [f32(e[1]) + f32(0.0) for e in ends]"),
    "ends_only_without_epsilon": ("        if j == Tp:\n            ends.append((s, c, words))",
                                  "        if j == Tp and not out_arcs.get((j, s)):\n            ends.append((s, c, words))"),
    "worst_not_best": ("if words not in best or t < best[words]:", "if words not in best or t > best[words]:"),
}


def run_pins(mod):
    pins.WL = mod
    try:
        for seed in range(12):
            pins.test_best_word_sequence_is_the_decode_best_path(seed)
            pins.test_whole_lattice_holds_every_path_of_the_graph(seed)
        pins.test_kept_frames_of_label_synchronous_decoding()
        pins.test_without_output_labels_one_empty_sequence()
        pins.test_pruned_lattice_is_a_subset()
    finally:
        import oracle.word_lattice as real
        pins.WL = real


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert old in src, "mutation anchor missing: " + name
    # the first occurrence: the lattice map the pins check against the decoder
    path = tmp_path / "word_lattice_mut.py"
    path.write_text(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location("word_lattice_mut", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    with pytest.raises((AssertionError, ValueError, IndexError, KeyError)):
        run_pins(mod)


def test_unmutated_module_passes():
    import oracle.word_lattice as real
    run_pins(real)
