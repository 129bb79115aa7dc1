"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle.

Random numbers only: shapes, masks, bit plans, weights, activations and router
logits.  None of the layer's arithmetic lives here."""
