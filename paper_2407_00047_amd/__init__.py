"""QLM batched request-waiting-time estimation and SLO-violation scoring of
candidate virtual-queue plans, on MI355X (gfx950)."""
