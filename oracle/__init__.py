"""CPU oracle for the boosted-decode hot path — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run anything in this package. The product path
(``paper_2608_21343_amd``) never calls it and shares no code with it: the two
meet only in the seeded input generators of ``workloads``.

What it computes (TurboBias 2.0, Sec. II):

* ``graph.build_graph``: one phrase list -> a case-insensitive boosting graph.
  Phrases are mapped to case-class strings (Sec. II-A: matching must not
  depend on the emitted capitalization), merged into a dictionary trie, and
  given textbook Aho-Corasick failure (suffix) links (Sec. II-A/II-B: the
  boosting structure is a tree with suffix links). State potentials phi, end
  bonuses E and psi = phi + E follow the potential-difference scoring of
  Sec. II-A (an arc scores phi(dst) - phi(src)).
* ``decode.greedy_decode`` / ``decode.beam_decode``: per-stream boosted
  greedy and beam steps over joint-logit rows (Sec. II-B: each stream carries a
  model id, -1 meaning no biasing; Sec. II-C: state carried across chunks).
* ``variative.build_variative_graph``: the case-insensitive variative BPE
  graph of Sec. II-A (Fig. 1c, 1e) over a piece vocabulary, with the Eq. (1)
  split of each backbone token's score over its characters, encoded as one
  state per arc so that the same steps decode it.
* ``decode.beam_decode_stream``: the streaming beam of Sec. II-C with
  hypothesis recombination (equal label sequences merged by log-add-exp) and a
  flattened tree of the kept label records.

Floating point: potentials are computed in float64 and rounded once to
float32. Keys, beam candidates and accumulated beam scores are float32 with a
fixed operation order, because they decide integer outputs (argmax, top-K)
and the GPU takes the same decisions in float32. The log-softmax normalizer
is computed in float64 (exact summation) and rounded once to float32.

Pins (tests/test_oracle_*.py): brute-force suffix enumeration for the graph
states, hand-derived worked examples for the potentials (tests/golden/),
closed forms for the log-softmax normalizer and the pure-potential reading,
exhaustive enumeration for tiny beams, and invariants stated by the paper
(case invariance, model -1 equals unbiased decoding, per-stream isolation,
chunk invariance).
"""

from .graph import Graph, build_graph  # noqa: F401
from .variative import build_variative_graph, class_map_of, eq1_split  # noqa: F401
from .decode import (  # noqa: F401
    beam_decode,
    beam_decode_stream,
    greedy_decode,
    init_carry,
    init_stream_carry,
    lse32,
    tree_sequence,
    widen,
)
