"""Aladdin SLO- and KV-aware query placement evaluator for MI355X (gfx950)."""
