"""CPU oracle for the training step of dynamic-control-flow models.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or
executes this package; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.

The oracle is the imperative program itself, written plainly in numpy
float64: a Python loop over time steps and layers for the LSTM (the loop of
Figure 1, whose trip count depends on the data, Section 4.2.1), a recursive
walk over tree nodes for the TreeLSTM (the recursive calls of Section 4.2.1
and footnote 6), and hand-derived backward passes (the automatic
differentiation the paper inserts into the graph, Section 3.1).  Converting
such a program to a graph must not change its result (Section 3.2: the graph
is only used while its assumptions hold), so the oracle is the plain
definition of what the device path computes, not an approximation of it.

The paper does not define the cell equations; it names the models it trains
(Section 6.1, Table 2: LSTM [51], LM [21], TreeLSTM [40]).  The equations
used here are the standard ones of those models, stated in each module.
"""
from . import childsum, heads, lstm, schedule, sgd, steps, treelstm, treernn  # noqa: F401
